"""Benchmark: batched what-if evaluation of DVFS frequency policies on one MI355X.

One step is the whole hot path over one batch of candidate policies: one emo_evaluate launch
that computes, for every candidate, the forward pass (finish times, makespan, energy), the
backward pass (slack of every pack) when the workload has it, and the feasibility mask and
least-energy feasible candidate under the latency target; workloads with two targets take both
from that one launch (emo_evaluate_targets: every target's mask bits and selection records from
the evaluating kernel, one finalize launch for all of them).

By default all five workloads run one after another.  The headline is the largest one that fits
one GPU, the per-kernel graph of 65,536 kernels and 65,536 host nodes (2^14 candidates,
forward and backward for every candidate); the other four are reported under "configs".
Inputs are resident in HBM before timing starts; level batches that fit rotate over several
copies so that the 256 MB last-level cache does not hold them across steps.

Prints one JSON line.  `value` is candidate policies fully evaluated per second.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "candidate policies evaluated/sec (timing+energy+select); % of VALU/HBM roofline"
HEADLINE = 5            # the largest workload: 65,536 kernels + 65,536 host nodes, slack
HBM_PEAK_GBS = 8000.0
VALU_PEAK_TOPS = 39.3   # 256 CUs x 64 fp32 lanes x 2.4 GHz, one op per lane per clock (no packed math)


# sources that make the kernels of each kind (last_kernels): graph preparation and the
# selection code are common to all of them
KIND_SOURCES = {0: ("emo_kernels.hip",), 1: ("emo_jit.cpp",), 2: ("emo_jit.cpp",),
                3: ("emo_chains.hip", "emo_kernels.hip"), 4: ("emo_chains.hip", "emo_kernels.hip"),
                5: ("emo_jit.cpp",), 6: ("emo_chains.hip", "emo_kernels.hip"),
                7: ("emo_jit.cpp",), 8: ("emo_chains.hip", "emo_kernels.hip")}


def kernel_source_hash(kind: int) -> str:
    """Hash of the sources that generate the kernels of `kind`, so that a committed counter
    summary goes stale only when the kernel it measured can have changed."""
    h = hashlib.sha256()
    for name in KIND_SOURCES[kind] + ("emo_internal.h", "emo_host.cpp", "emo_select.h"):
        with open(os.path.join(ROOT, "paper_2607_12324_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload_name: str, kernel: str, src_hash: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary (FETCH_SIZE and
    WRITE_SIZE scaled by a plain copy's readings), or None when the kernel sources changed
    since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload_name}_traffic.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line:
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("source_hash") != src_hash:
        return None
    return float(fields["hbm_bytes_per_launch"])


def host_cpu():
    """Host facts for the CPU baseline: logical CPUs, the CPUs this process may run on, the
    threads the baseline uses (the box's share: OMP_NUM_THREADS, else the affinity set) and the
    CPU model."""
    n_aff = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or n_aff
    threads = max(1, min(threads, n_aff))
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "affinity": n_aff, "threads": threads, "model": model}


def cpu_baseline(k, g, rows, out, targets, budget_s: float = 20.0):
    """The oracle (plain fp64 C) on the host: the whole candidate batch (or, beyond the budget,
    a leading prefix) on all the threads this process may use, doing the step's work per
    candidate (makespan and energy, slack of every pack when the step has it, the selection
    for each target), then a bounded one-thread run.  The oracle's outputs are compared with
    the step's device outputs `out` (parity statistics); only the oracle calls are timed."""
    import numpy as np

    import oracle
    from paper_2607_12324_amd import emo, synth
    oracle.build()
    spec = synth.CONFIGS[k]
    B, P = rows.shape
    hc = host_cpu()
    nt = hc["threads"]
    # pieces of at most 2^27 slack values (1 GiB of fp64) or 2^16 rows
    step = max(1, min(1 << 16, (1 << 27) // max(1, P))) if spec.slack else 1 << 18
    T_or = np.empty(B)
    E_or = np.empty(B)
    t_oracle = 0.0
    done = 0
    s_max_err, s_bad, s_rows = 0.0, 0, 0
    while done < B:
        n = min(step, B - done)
        blk = rows[done:done + n]
        t = time.perf_counter()
        if spec.slack:
            T_b, E_b, S_b = oracle.slack_batch(g, blk, nthreads=nt)
        else:
            T_b, E_b = oracle.eval_batch(g, blk, nthreads=nt)
        t_oracle += time.perf_counter() - t
        T_or[done:done + n], E_or[done:done + n] = T_b, E_b
        if spec.slack:
            S_d = out["S"][done:done + n].cpu().numpy().astype(np.float64)
            ok = ~np.isnan(S_b)
            s_bad += int(np.count_nonzero(np.isnan(S_d) != ~ok))
            err = np.abs(S_d[ok] - S_b[ok]) / np.repeat(np.maximum(T_b, 1e-30), P).reshape(n, P)[ok]
            s_max_err = max(s_max_err, float(err.max()) if err.size else 0.0)
            s_rows += n
            del S_d, S_b
        done += n
        if t_oracle > budget_s:
            break
    n_or = done
    t = time.perf_counter()
    sels = [oracle.select(T_or[:n_or], E_or[:n_or], tgt) for tgt in targets]
    t_oracle += time.perf_counter() - t
    # parity of the step's outputs over the rows the oracle evaluated
    Td = out["T"][:n_or].cpu().numpy().astype(np.float64)
    Ed = out["E"][:n_or].cpu().numpy().astype(np.float64)
    parity = {"rows": n_or, "of": B,
              "makespan_max_rel_err": float(np.max(np.abs(Td - T_or[:n_or]) / T_or[:n_or])),
              "makespan_mismatches": int(np.count_nonzero(Td != T_or[:n_or])),
              "energy_max_rel_err": float(np.max(np.abs(Ed - E_or[:n_or]) / E_or[:n_or]))}
    if spec.slack:
        parity.update({"slack_rows": s_rows, "slack_max_err_over_makespan": s_max_err,
                       "slack_nan_mismatches": s_bad})
    agree = []
    for tgt, (idx, feas, nf), m, r in zip(targets, sels, out["masks"], out["results"]):
        if n_or == B:
            bits = emo.unpack_mask(m, B)
            sel = emo.parse_selection(r)
        else:   # a prefix: re-select the device outputs over the same prefix
            r2, m2 = emo.select_from_results(out["T"][:n_or], out["E"][:n_or], tgt)
            bits, sel = emo.unpack_mask(m2, n_or), emo.parse_selection(r2)
        best = E_or[idx] if idx >= 0 else np.nan
        near = feas & (np.abs(E_or[:n_or] - best) <= 1e-5 * best) if idx >= 0 else feas & False
        agree.append({"target": tgt, "oracle_index": idx, "index": sel.index,
                      "agree": bool(sel.index == idx or (idx >= 0 and 0 <= sel.index < n_or and near[sel.index])),
                      "oracle_feasible": nf, "feasible": sel.num_feasible,
                      "mask_mismatches": int(np.count_nonzero(bits != feas))})
    parity["selection"] = agree
    # one thread on a bounded prefix
    n1 = max(1, min(B, int(n_or / max(t_oracle, 1e-9) / nt * 2.0)))
    t = time.perf_counter()
    if spec.slack:
        oracle.slack_batch(g, rows[:n1], nthreads=1)
    else:
        oracle.eval_batch(g, rows[:n1], nthreads=1)
    t1 = time.perf_counter() - t
    what = "makespan + energy + slack of every pack" if spec.slack else "makespan + energy"
    base = {"value": n_or / t_oracle, "unit": "policies/s", "cores": nt, "kind": "oracle",
            "sample": (f"{'the whole batch' if n_or == B else f'the first {n_or} of {B} candidates'} "
                       f"({what}, selection at {len(targets)} target(s); fp64 C) on {nt} threads "
                       f"in {t_oracle:.2f} s"),
            "host": hc,
            "one_thread": {"value": n1 / t1, "unit": "policies/s", "cores": 1,
                           "sample": f"the first {n1} candidates, {what}, in {t1:.2f} s"}}
    return base, parity


def run_dp(args, emo, synth, np, torch):
    """Policy search (Alg. 2, one frequency interval per pack) on workload k's graph and tables:
    target 1.05 T0, buckets of 0.05 T0 / dp_buckets.  `value` = searches per second; the CPU
    baseline runs the search oracle (the fp64 C predictor under Python control, one thread) on
    the same search, whole when it takes seconds, else its first stages scaled to all stages."""
    k = args.workload
    g = synth.config_graph(k)
    P, F = g.num_packs, g.num_levels
    gh = emo.EmoGraph(g, device=0)
    top = torch.full((1, P), F - 1, dtype=torch.uint8, device="cuda")
    fast = torch.from_numpy(np.argmin(g.pack_time, axis=1).astype(np.uint8)[None, :]).cuda()
    T0 = float(gh.eval_policies(top)[0].item())
    Tl = float(gh.eval_policies(fast)[0].item())
    tgt = float(np.float32(1.05 * T0))
    q = float(np.float32(0.05 * T0 / args.dp_buckets))
    nb = int(np.floor(tgt / q)) - max(0, int(np.floor(Tl / q)) - 1) + 1
    cands = 1 + F + max(P - 1, 0) * nb * F
    lv, res = gh.dp_search(tgt, q)
    for _ in range(max(args.warmup - 1, 0)):
        gh.dp_search(tgt, q, best_levels=lv, result=res)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    a.record()
    for _ in range(args.steps):
        gh.dp_search(tgt, q, best_levels=lv, result=res)
    b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms = a.elapsed_time(b) / args.steps
    sel = emo.parse_selection(res)
    E0 = float(gh.eval_policies(top)[1].item())
    out = {
        "metric": "policy search (Alg. 2, one interval per pack): searches/sec",
        "value": 1e3 / ms, "unit": "searches/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": synth.CONFIGS[k].name, "packs": P, "levels": F, "stages": P,
                   "buckets": nb, "quantum": q, "target_ratio": 1.05,
                   "candidates_per_search": cands, "step": "emo_dp_search"},
        "per_stage_us": 1e3 * ms / max(P, 1),
        "candidates_evaluated_per_s": cands / (ms / 1e3),
        "roofline": None,
        "roofline_note": "launch-bound: a stage evaluates at most buckets x levels candidates "
                         "(a few MB) in one evaluation kernel plus two small kernels",
        "result": {"energy": sel.energy, "makespan": sel.makespan, "bucket": sel.index,
                   "states": sel.num_feasible, "all_max_energy": E0, "T0": T0},
        "wall_s": wall,
    }
    if not args.no_cpu_baseline:
        from oracle import dp as odp   # the CPU baseline leg only
        stages = P if P * nb * F <= 1 << 20 else max(1, (1 << 20) // (nb * F))
        t = time.perf_counter()
        r = odp.dp_search(g, tgt, q, max_stages=stages)
        dt = time.perf_counter() - t
        whole = stages == P
        out["cpu_baseline"] = {"value": stages / (dt * P), "unit": "searches/s", "cores": 1,
                               "kind": "oracle",
                               "sample": (f"the whole search ({r.evaluated} candidate evaluations in {dt:.2f} s"
                                          if whole else
                                          f"the first {stages} of {P} stages ({r.evaluated} candidate "
                                          f"evaluations in {dt:.2f} s), scaled to {P} stages")
                                         + "; fp64 C predictor, Python control, 1 thread)",
                               "result": ({"energy": r.energy, "makespan": r.makespan,
                                           "states": r.num_states} if whole else None)}
    print(json.dumps(out), flush=True)


def run_pack(args, emo, synth, np, torch):
    """Dependency-aware greedy packing (emo_pack_kernels + emo_contract_packs, host passes) of
    workload k's graph with every pack taken as one kernel, bound 5 ms.  `value` = packings per
    second; beside it the packed graph's evaluation rate (emo_evaluate on the workload's number
    of candidates) next to the per-kernel graph's, and the packing oracle on the host."""
    k = args.workload
    spec = synth.CONFIGS[k]
    g = synth.config_graph(k)
    bound = 5000.0
    times = []
    for i in range(args.warmup + args.steps):
        t = time.perf_counter()
        grp, n = emo.pack_kernels(g, g.node_stream, bound)
        pg = emo.contract_packs(g, grp, n)
        if i >= args.warmup:
            times.append(time.perf_counter() - t)
    ms = 1e3 * float(np.median(times))
    F, B = g.num_levels, spec.num_candidates

    def eval_rate(graph, rows):
        gh = emo.EmoGraph(graph, device=0)
        lv = torch.from_numpy(rows).cuda()
        T = torch.empty(B, dtype=torch.float32, device="cuda")
        E = torch.empty_like(T)
        for _ in range(3):
            gh.eval_policies(lv, T, E)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record()
        reps = 5
        for _ in range(reps):
            gh.eval_policies(lv, T, E)
        b.record()
        torch.cuda.synchronize()
        t0 = float(T[0].item())
        gh.close()
        return B / (a.elapsed_time(b) / reps / 1e3), t0

    rng = np.random.default_rng(spec.policy_seed)
    rows = rng.integers(0, F, (B, n)).astype(np.uint8)
    rows[0] = F - 1
    kernel_rows = np.ascontiguousarray(rows[:, grp])
    packed_rate, T0p = eval_rate(pg, rows)
    unpacked_rate, T0u = eval_rate(g, kernel_rows)
    out = {
        "metric": "dependency-aware greedy packing (Sec. IV-D), host pass: packings/sec",
        "value": 1e3 / ms, "unit": "packings/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": spec.name, "kernels": g.num_packs, "nodes": g.num_nodes,
                   "edges": g.num_edges, "max_pack_duration_us": bound,
                   "step": "emo_pack_kernels + emo_contract_packs"},
        "packed": {"packs": n, "nodes": pg.num_nodes, "edges": pg.num_edges,
                   "all_max_makespan_packed": T0p, "all_max_makespan_per_kernel": T0u,
                   "eval_policies_per_s_packed": packed_rate,
                   "eval_policies_per_s_per_kernel": unpacked_rate, "candidates": B},
        "roofline": None,
        "roofline_note": "host pass, O(V + E) once per graph; no device kernel",
    }
    if not args.no_cpu_baseline:
        from oracle import packing as opk   # the CPU baseline leg only
        t = time.perf_counter()
        og, on = opk.pack_kernels(g, g.node_stream, bound)
        opk.contract(g, og, on)
        dt = time.perf_counter() - t
        out["cpu_baseline"] = {"value": 1.0 / dt, "unit": "packings/s", "cores": 1,
                               "kind": "oracle",
                               "sample": "one whole packing and contraction of the same graph "
                                         "(Python over the fp64 C schedule, 1 thread)",
                               "same_result": bool(on == n and np.array_equal(og, grp))}
    print(json.dumps(out), flush=True)


def run_model(args, emo, synth, np, torch):
    """Microbenchmark pack model (emo_pack_model, host pass, Eq. 6-7) for every pack of workload
    k: a 16-metric, 12-benchmark suite; `value` = packs modelled per second.  The CPU baseline
    runs the pack-model oracle on the first packs for about 10 s."""
    k = args.workload
    g = synth.config_graph(k)
    mi = synth.model_inputs(k, g.num_packs, g.num_levels)
    times = []
    for i in range(args.warmup + args.steps):
        t = time.perf_counter()
        W, T, E = emo.pack_model(mi.metric_matrix, mi.bench_time, mi.bench_energy, mi.pack_metrics)
        if i >= args.warmup:
            times.append(time.perf_counter() - t)
    ms = 1e3 * float(np.median(times))
    threads = os.cpu_count()
    out = {
        "metric": "microbenchmark pack model (Sec. IV-E, NNLS + Eq. 7), host pass: packs/sec",
        "value": g.num_packs / (ms / 1e3), "unit": "packs/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": synth.CONFIGS[k].name, "packs": g.num_packs,
                   "levels": g.num_levels, "metrics": int(mi.metric_matrix.shape[0]),
                   "benchmarks": int(mi.metric_matrix.shape[1]), "host_threads": threads,
                   "step": "emo_pack_model"},
        "roofline": None,
        "roofline_note": "host pass, once per graph; no device kernel",
    }
    if not args.no_cpu_baseline:
        from oracle import pack_model as opm   # the CPU baseline leg only
        t = time.perf_counter()
        done = 0
        same = True
        while done < g.num_packs and time.perf_counter() - t < 10.0:
            x, _ = opm.fit_pack(mi.metric_matrix, mi.pack_metrics[done])
            to, _ = opm.predict(x, mi.bench_time, mi.bench_energy)
            same &= bool(np.allclose(to, T[done], rtol=1e-6))
            done += 1
        dt = time.perf_counter() - t
        out["cpu_baseline"] = {"value": done / dt, "unit": "packs/s", "cores": 1, "kind": "oracle",
                               "sample": f"the first {done} packs ({dt:.1f} s; SciPy NNLS certified "
                                         "by KKT, Eq. 7 in Python, 1 thread)",
                               "same_tables": same}
    print(json.dumps(out), flush=True)


def run_intervals(args, emo, synth, np, torch):
    """Time-interval policies (emo_eval_intervals) on workload k's graph: the workload's batch
    size, K intervals over [0, 1.05 T0) (change points on the time grid), idle power rising with
    the level's frequency, uniform random levels; one call per step with mask and selection at
    1.02 T0.  `value` = candidates per second."""
    k = args.workload
    spec = synth.CONFIGS[k]
    g = synth.config_graph(k)
    F, K, B = g.num_levels, args.intervals, spec.num_candidates
    gh = emo.EmoGraph(g, device=0)
    dev = torch.device("cuda", 0)
    top = torch.full((1, g.num_packs), F - 1, dtype=torch.uint8, device=dev)
    T0 = float(gh.eval_policies(top)[0].item())
    pts = [float(synth.quantize(T0 * 1.05 * (i + 1) / K)) for i in range(K - 1)]
    idle = [float(x) for x in np.round(g.static_power * (0.5 + 0.5 * synth.level_ratios(F)) * 64) / 64]
    rows = synth.random_policies_parallel(spec.policy_seed, K, F, B, "uniform", workers=8)
    copies = max(1, args.copies if B * K < (1 << 30) else 1)
    lv = [torch.from_numpy(rows).to(dev)]
    for _ in range(copies - 1):
        lv.append(lv[0].clone())
    T = torch.empty(B, dtype=torch.float32, device=dev)
    E = torch.empty(B, dtype=torch.float32, device=dev)
    m = torch.empty((B + 31) // 32, dtype=torch.int32, device=dev)
    r = torch.empty(3, dtype=torch.int64, device=dev)
    tgt = float(np.float32(1.02 * T0))
    stream = torch.cuda.current_stream()

    def call(i):
        gh.eval_intervals(lv[i % copies], pts, idle, makespan=T, energy=E, latency_target=tgt, mask=m,
                          result=r)

    for i in range(args.warmup):
        call(i)
    torch.cuda.synchronize()
    every = max(1, args.time_every)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(0, args.steps, every)]
    for a, b in ev:
        a.record(stream)
        b.record(stream)
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record(stream)
    for i in range(args.steps):
        if i % every == 0:
            gh.set_timing_events(ev[i // every][0], ev[i // every][1])
        elif i % every == 1:
            gh.set_timing_events(None, None)
        call(i)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    gh.set_timing_events(None, None)
    ms_step = start.elapsed_time(end) / args.steps
    main_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    info = gh.info()
    algo_bytes = B * (K + 8) + (B + 7) // 8
    achieved = algo_bytes / (main_ms / 1e3) / 1e9
    # per candidate: the forward work of the per-pack kernel plus, per pack, the binary search
    # over the change points (one compare and one select per halving step)
    steps = int(np.ceil(np.log2(K))) if K > 1 else 0
    ops_per_cand = info["num_dynamic_edges"] + 2 * g.num_packs + 2 + 2 * steps * g.num_packs + 3 * K
    valu_tops = B * ops_per_cand / (main_ms / 1e3) / 1e12
    sel = emo.parse_selection(r)
    out = {
        "metric": "time-interval policies evaluated/sec (makespan + energy + selection)",
        "value": B / (ms_step / 1e3), "unit": "policies/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": spec.name, "candidates": B, "intervals": K, "packs": g.num_packs,
                   "levels": F, "target_ratio": 1.02, "step": "emo_eval_intervals",
                   "rotated_input_copies": copies, "kernels": info["last_kernels"]},
        "roofline": {"bound": "hbm",
                     "kernel": "emo_iv" if info["last_kernels"] == 7
                     else "interval_kernel", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": None, "algorithmic_bytes_per_launch": algo_bytes,
                     "launch_ms": main_ms, "timed_launches": len(ev),
                     "valu": {"achieved": valu_tops, "peak": VALU_PEAK_TOPS, "unit": "Tops/s",
                              "frac": valu_tops / VALU_PEAK_TOPS,
                              "algorithmic_ops_per_candidate": ops_per_cand}},
        "selected": {"index": sel.index, "energy": sel.energy, "makespan": sel.makespan,
                     "num_feasible": sel.num_feasible},
        "wall_s": wall,
    }
    if not args.no_cpu_baseline:
        from oracle import intervals as oiv   # the CPU baseline leg only
        n = 2048
        t = time.perf_counter()
        oiv.eval_intervals(g, pts, rows[:n], idle)
        dt = time.perf_counter() - t
        out["cpu_baseline"] = {"value": n / dt, "unit": "policies/s", "cores": 1, "kind": "oracle",
                               "sample": f"the first {n} candidates of the batch in {dt:.2f} s "
                                         "(pure-Python fp64 interval oracle, 1 thread)"}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=0,
                    help="one benchmark workload 1..5; default 0: all five, the largest "
                         "(65,536 kernels) as the headline and the others under 'configs'")
    ap.add_argument("--copies", type=int, default=5, help="rotated copies of the level batch")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the graph variants of the default run (4096-pack graph off the time "
                         "grid and without cut nodes, 65,536-kernel graph off the grid)")
    ap.add_argument("--time-every", type=int, default=8,
                    help="time the main launch with a HIP event pair on every N-th timed step "
                         "(an event record costs a few microseconds of device time; default 8)")
    ap.add_argument("--dp", action="store_true",
                    help="time the policy search of Alg. 2 (emo_dp_search) on the workload's graph "
                         "instead of the evaluation step")
    ap.add_argument("--intervals", type=int, default=0, metavar="K",
                    help="time emo_eval_intervals (time-interval policies with K intervals) on the "
                         "workload's graph and batch size instead of the evaluation step")
    ap.add_argument("--pack", action="store_true",
                    help="time the packing pass on --workload's graph (each pack one kernel)")
    ap.add_argument("--model", action="store_true",
                    help="time the pack model (NNLS, Eq. 7) for every pack of --workload")
    ap.add_argument("--dp-buckets", type=int, default=64,
                    help="makespan buckets of the search between T0 and 1.05 T0 (default 64)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB, --steps times (the reference "
                         "kernel for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the library evaluates candidate policies on a single "
              "MI355X (candidates would shard across GPUs with one MIN all-reduce of the "
              "selection key; that path is not built).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_12324_amd import emo, synth

    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "launches": args.steps}))
        return

    if (args.dp or args.intervals or args.pack or args.model) and args.workload == 0:
        args.workload = 2
    if args.dp:
        run_dp(args, emo, synth, np, torch)
        return
    if args.intervals:
        run_intervals(args, emo, synth, np, torch)
        return
    if args.pack:
        run_pack(args, emo, synth, np, torch)
        return
    if args.model:
        run_model(args, emo, synth, np, torch)
        return

    ks = [1, 2, 3, 4, 5] if args.workload == 0 else [args.workload]
    head = HEADLINE if args.workload == 0 else args.workload
    recs = {}
    t_all = time.perf_counter()
    for k in ks:
        recs[k] = run_workload(k, args, emo, synth, np, torch)
        print(f"# workload {k} done: {recs[k]['ms_per_step']:.4f} ms/step, "
              f"{recs[k]['value']:.4g} policies/s", file=sys.stderr, flush=True)
    # the 4096-pack workload's graph off the exact-sum time grid (cut-segment kernels, segment-
    # local rounding) and without cut nodes (segmented kernels), and the 65,536-kernel graph off
    # the grid (chain scan, prefix-sum rounding): the same steps and batches
    variants = {}
    if args.workload == 0 and not args.no_variants:
        g4, g5 = synth.config_graph(4), synth.config_graph(5)
        for k, gv in ((4, synth.scaled_times(g4, 1.1)), (4, synth.without_cuts(g4)),
                      (5, synth.scaled_times(g5, 1.1))):
            r = run_workload(k, args, emo, synth, np, torch, graph=gv, cpu_budget_s=3.0)
            print(f"# variant {gv.name} done: {r['ms_per_step']:.4f} ms/step", file=sys.stderr, flush=True)
            variants[gv.name] = {x: r.get(x) for x in ("value", "ms_per_step", "config", "roofline", "kernels",
                                                       "parity", "compile_seconds", "selected")}
    h = recs[head]
    out = {
        "metric": METRIC,
        "value": h["value"],
        "unit": "policies/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": h["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": h["config"],
        "roofline": h["roofline"],
        "cpu_baseline": h.get("cpu_baseline"),
        "parity": h.get("parity"),
        "selected": h["selected"],
        "compile_seconds": h["compile_seconds"],
        "hip_runtime_version": h["hip_runtime_version"],
        "kernel_source_hash": h["kernel_source_hash"],
        "configs": {synth.CONFIGS[k].name: {x: v for x, v in recs[k].items() if x != "config"} |
                    {"config": recs[k]["config"]} for k in ks if k != head},
        "variants": variants,
        "wall_s": time.perf_counter() - t_all,
    }
    print(json.dumps(out), flush=True)


def run_workload(k, args, emo, synth, np, torch, graph=None, cpu_budget_s=20.0):
    """One workload's step timed over args.steps steps (after args.warmup), its roofline, and,
    unless disabled, the oracle baseline with parity statistics.  Frees its device memory.
    `graph`: a variant of the workload's graph (same packs and levels) to run instead; its
    traffic is not looked up (the committed counters are the workload's own graph's)."""
    spec = synth.CONFIGS[k]
    g = synth.config_graph(k) if graph is None else graph
    B = spec.num_candidates
    P = g.num_packs
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    rows = synth.bench_policies(k, g)
    copies = max(1, args.copies if B * P < (1 << 30) else 1)
    lv = [torch.from_numpy(rows).to(dev)]
    for _ in range(copies - 1):
        lv.append(lv[0].clone())
    gh = emo.EmoGraph(g, device=0)
    stream = torch.cuda.current_stream()
    T = torch.empty(B, dtype=torch.float32, device=dev)
    E = torch.empty(B, dtype=torch.float32, device=dev)
    S = torch.empty((B, P), dtype=torch.float32, device=dev) if spec.slack else None
    masks = [torch.empty((B + 31) // 32, dtype=torch.int32, device=dev) for _ in spec.targets]
    res_all = torch.empty((len(spec.targets), 3), dtype=torch.int64, device=dev)
    results = [res_all[j] for j in range(len(spec.targets))]
    t_c = time.perf_counter()
    T0, _ = gh.eval_policies(lv[0][:1])       # row 0 is the all-max policy
    targets = [float(np.float32(r * float(T0.item()))) for r in spec.targets]

    def main_call(x):
        if len(targets) == 1:
            gh.evaluate(x, makespan=T, energy=E, slack=S, latency_target=targets[0], mask=masks[0],
                        result=results[0])
        else:
            # every target's mask and selection records from the one evaluating launch
            gh.evaluate_targets(x, targets, makespan=T, energy=E, slack=S, masks=masks, results=res_all)

    def step(i):
        main_call(lv[i % copies])

    step(0)                                   # compiles the specialised kernels if any
    torch.cuda.synchronize()
    first_call_s = time.perf_counter() - t_c
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    def timed(copies_used):
        every = max(1, args.time_every)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(0, args.steps, every)]
        for a, b in ev:   # create the underlying HIP events
            a.record(stream)
            b.record(stream)
        start = torch.cuda.Event(enable_timing=True)
        end = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t_wall = time.perf_counter()
        start.record(stream)
        for i in range(args.steps):
            # the library records the pair right around the kernel(s) evaluating the candidates
            if i % every == 0:
                gh.set_timing_events(ev[i // every][0], ev[i // every][1])
            elif i % every == 1:
                gh.set_timing_events(None, None)
            main_call(lv[i % copies_used])
        end.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t_wall
        gh.set_timing_events(None, None)
        return (start.elapsed_time(end) / args.steps,
                float(np.mean([a.elapsed_time(b) for a, b in ev])), len(ev), wall)

    ms_step, main_ms, n_ev, wall = timed(copies)
    cache = None
    if copies > 1:
        # the same step on one resident input copy (a small batch then stays in the 256 MB
        # last-level cache across steps)
        ms1, main1, _, _ = timed(1)
        cache = {"ms_per_step": ms1, "value": B / (ms1 / 1e3), "launch_ms": main1}
    sels = [emo.parse_selection(r) for r in results]
    info = gh.info()

    value = B / (ms_step / 1e3)
    # algorithmic bytes of the main launch: level bytes in; makespan, energy, slack and mask out
    algo_bytes = B * (P + 8 + (4 * P if spec.slack else 0)) + len(targets) * ((B + 7) // 8)
    achieved = algo_bytes / (main_ms / 1e3) / 1e9
    # algorithmic VALU work on the folded graph: one max per candidate-dependent edge, one add
    # per pack for the finish time and one for the energy, two for the makespan/energy close;
    # the backward pass (min per edge, subtractions per node) doubles it
    ops_per_cand = (info["num_dynamic_edges"] + 2 * P + 2) * (2 if spec.slack else 1)
    valu_tops = B * ops_per_cand / (main_ms / 1e3) / 1e12
    src_hash = kernel_source_hash(info["last_kernels"])
    kname = kernel_name(info["last_kernels"], spec.slack)
    traffic = measured_traffic(spec.name, kname, src_hash) if graph is None else None
    rec = {
        "value": value,
        "ms_per_step": ms_step,
        "config": {"workload": g.name, "candidates": B, "nodes": g.num_nodes,
                   "edges": g.num_edges, "packs": P, "levels": g.num_levels,
                   "target_ratios": list(spec.targets), "slack": spec.slack,
                   "step": "emo_evaluate" if len(targets) == 1 else f"emo_evaluate_targets ({len(targets)} targets)",
                   "rotated_input_copies": copies},
        "roofline": {"bound": "hbm", "kernel": kname, "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic,
                     "traffic_ratio": None if traffic is None else traffic / algo_bytes,
                     "algorithmic_bytes_per_launch": algo_bytes,
                     "launch_ms": main_ms, "timed_launches": n_ev,
                     "valu": {"achieved": valu_tops, "peak": VALU_PEAK_TOPS, "unit": "Tops/s",
                              "frac": valu_tops / VALU_PEAK_TOPS,
                              "algorithmic_ops_per_candidate": ops_per_cand}},
        "cache_resident": cache,
        "selected": [{"target": t, "index": x.index, "energy": x.energy, "makespan": x.makespan,
                      "num_feasible": x.num_feasible} for t, x in zip(targets, sels)],
        "kernels": info["last_kernels"],
        "compile_seconds": info["compile_seconds"],
        "first_call_s": first_call_s,
        "hip_runtime_version": info["hip_runtime_version"],
        "kernel_source_hash": src_hash,
        "timed_wall_s": wall,
    }
    if not args.no_cpu_baseline:
        out = {"T": T, "E": E, "S": S, "masks": masks, "results": results}
        rec["cpu_baseline"], rec["parity"] = cpu_baseline(k, g, rows, out, targets, budget_s=cpu_budget_s)
    del lv, S, T, E, rows
    gh.close()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return rec


def kernel_name(kind: int, slack: bool) -> str:
    """The evaluating kernel (or chain of kernels timed as one unit) of a kernel kind."""
    return {2: "emo_chain", 3: "chains_kernel", 4: "chains_windowed", 5: "emo_cut", 6: "chains_scan", 8: "chains_scan_full",
            1: "emo_sp_slack" if slack else "emo_sp_select"}.get(
                kind, "slack_kernel" if slack else "forward_kernel")

if __name__ == "__main__":
    main()
