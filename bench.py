#!/usr/bin/env python3
"""Throughput of the cache-aware MoE decode step on one MI355X.

One step = one decode token for every stream through all L MoE layers in
causal order (router GEMV, cache step, residency and fills, expert FFN).  The
default workload is the Qwen3-30B-A3B-shaped bf16 slice (L=48, N=128, K=8,
d=2048, SwiGLU 2048->768->2048, C=32, update-only Temporal Router, 64 streams
x 512 tokens, AR(1) hidden states); all inputs are synthetic, seeded and
resident in HBM before the timed region.  The metric is token-layer steps per
second: streams x layers x timed tokens / time.

Prints one JSON line.  The timed region launches the decode path and nothing
else.  Besides the throughput the line carries the roofline of the dominant
kernel (expert gate/up), whose average duration comes from HIP events that a
second pass of the same length attaches to each of its launches, the cache
statistics (Hit, AdjHit, Load/token), the CPU oracle's throughput on a bounded
sample (measured before the process touches the GPU) and, as context only, the
paper's own hit-rate and traffic figures.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PAPER_METRICS = os.path.join(ROOT, "tests", "golden", "paper_metrics.json")
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "ffn_up_bf16_qwen3_30b_traffic.md")


def measured_traffic(w):
    """HBM bytes per ffn_up launch from the committed rocprofv3 counter runs,
    or None if they were taken on another workload or on other kernel sources."""
    import hashlib
    if (w.name, w.mode, w.policy, w.C, w.R) != ("qwen3_30b", 0, 0, 32, 0) or not os.path.exists(TRAFFIC_PROFILE):
        return None
    vals = {}
    for line in open(TRAFFIC_PROFILE):
        if ":" in line and line.split(":")[0] in ("traffic_bytes_per_launch", "sources_sha256"):
            k, v = line.split(":", 1)
            vals[k] = v.strip()
    src = os.path.join(ROOT, "paper_2609_04895_amd", "csrc")
    digest = hashlib.sha256(open(os.path.join(src, "ffn.hip"), "rb").read()
                            + open(os.path.join(src, "fill.hip"), "rb").read()).hexdigest()
    if vals.get("sources_sha256") != digest:
        return None
    return float(vals["traffic_bytes_per_launch"])
METRIC = "cache-aware MoE decode token-layer steps/s per GPU; % HBM roofline; hit rate"


POLICIES = {"router": 0, "lru": 1, "lfu": 2, "lrfu": 3}
MODES = {"temporal": 0, "full": 1, "spatio_only": 2}


def describe(w):
    retention = {0: "Temporal Router", 1: "LRU", 2: "LFU", 3: f"LRFU(lambda={w.lrfu_lambda})"}[w.policy]
    mode = {0: f"update-only, {retention} retention", 1: f"full Spatio-Temporal, R={w.R}",
            2: f"Spatio-only, R={w.R}, {retention} retention"}[w.mode]
    dt = "bf16" if w.dtype == 1 else "fp32"
    import synth
    base_L = synth.WORKLOADS[w.name].L if w.name in synth.WORKLOADS else w.L
    layers = f"L={w.L}" if w.L == base_L else f"L={w.L} (the first {w.L} of its {base_L} layers)"
    return (f"{w.name}: {layers} N={w.N} K={w.K} d={w.d} SwiGLU {w.d}->{w.F}->{w.d} C={w.C} {mode}, "
            f"{w.S} streams x {w.T} tokens, {dt}, AR(1) rho={w.rho}"
            + (f", Zipf({w.zipf}) bias" if w.zipf else "")
            + (f", {w.arena_slots} HBM expert slots per layer" if w.arena_slots else ""))


def fills_label(w, fills):
    if not w.has_spatio or w.R == 0:
        return "none (no refinement)"
    return "side stream" if fills == "side" else "main stream, in the demand fill launch"


def cpu_baseline(w, budget_s, max_procs=16):
    """The oracle on stream 0, tokens 0.. until budget_s of oracle compute in
    one process; then the same tokens replayed by one process per host core
    at once (at most max_procs, the host share of one GPU), which gives its
    all-core rate on this workload.

    Must run before this process initialises the GPU: the all-core leg forks
    worker processes, which inherit the generated inputs and never touch the
    GPU.  Separate processes (not threads) keep one worker's Python glue from
    being timed as another's oracle work."""
    import multiprocessing

    import numpy as np

    import oracle
    import synth
    if "torch" in sys.modules and sys.modules["torch"].cuda.is_initialized():
        raise RuntimeError("cpu_baseline must run before the GPU is initialised (it forks)")
    kinds = [synth.KIND_ROUTER_NATIVE] + ([synth.KIND_ROUTER_TEMPORAL] if w.has_temporal else []) + \
        ([synth.KIND_ROUTER_SPATIO] if w.has_spatio else [])
    Ws = [[synth.router_host(w, k, l) for l in range(w.L)] for k in kinds]
    bias = synth.zipf_bias(w)
    Tmax = 64
    H = [synth.hidden_host(w, 0, l, T=Tmax) for l in range(w.L)]
    experts = {}

    def token(run, t, fetch):
        """One token through the oracle; returns its oracle seconds."""
        t0 = time.perf_counter()
        z = np.empty((len(kinds), 1, w.L, w.N), np.float32)
        for l in range(w.L):
            for r in range(len(kinds)):
                z[r, 0, l] = oracle.logits(Ws[r][l], H[l][t], bias[l] if (r == 0 and bias is not None) else None)
        out = run.step(z[0], z[1] if w.has_temporal else None, z[-1] if w.has_spatio else None)
        busy = time.perf_counter() - t0
        for l in range(w.L):
            sel = out["sel"][0, l]
            # host input generation and stacking are not oracle work: not timed
            ex = [fetch(l, int(e)) for e in sel]
            wg, wu, wd = (np.stack([x[i] for x in ex]) for i in range(3))
            t0 = time.perf_counter()
            oracle.moe_ffn(wg, wu, wd, out["gate"][0, l], H[l][t])
            busy += time.perf_counter() - t0
        return busy

    def generate(l, e):
        if (l, e) not in experts:
            experts[(l, e)] = synth.expert_host(w, l, e)
        return experts[(l, e)]

    def new_run():
        return oracle.Run(w.L, w.N, w.K, w.C, w.R, 1, w.mode, policy=w.policy, lrfu_lambda=w.lrfu_lambda)

    run = new_run()
    busy, tokens = 0.0, 0
    while tokens < Tmax and (tokens == 0 or busy < budget_s):
        busy += token(run, tokens, generate)
        tokens += 1
    affinity = len(os.sched_getaffinity(0))
    procs = min(max_procs, affinity)
    host = {"os_cpu_count": os.cpu_count(), "affinity_cores": affinity, "processes_used": procs,
            "cap": f"at most {max_procs} processes (the host share of one GPU)"}
    single = {"value": tokens * w.L / busy, "cores": 1,
              "sample": f"stream 0, tokens 0..{tokens - 1}, all {w.L} layers (router logits, cache step, "
                        f"SwiGLU FFN of the {w.K} selected experts), one process, {busy:.1f} s of oracle time"}
    res = {"value": single["value"], "unit": "token-layer steps/s", "cores": 1, "kind": "oracle",
           "sample": single["sample"], "host": host, "single_core": single}
    if procs > 1:
        # every worker replays the same tokens from a fresh state, so it
        # selects the same experts, all generated above and inherited
        ctx = multiprocessing.get_context("fork")
        start = ctx.Barrier(procs, timeout=300)
        results = ctx.Queue()

        def replay(i):
            try:
                r = new_run()
                start.wait()
                b = 0.0
                for t in range(tokens):
                    b += token(r, t, lambda l, e: experts[(l, e)])
                results.put((i, b, None))
            except Exception as exc:  # reported below; a failed worker breaks the barrier for the others
                start.abort()
                results.put((i, None, repr(exc)))

        pool = [ctx.Process(target=replay, args=(i,), daemon=True) for i in range(procs)]
        for p in pool:
            p.start()
        got = [results.get(timeout=900) for _ in range(procs)]
        for p in pool:
            p.join(timeout=60)
        errors = [e for _, _, e in got if e is not None]
        if errors:
            res["all_cores_error"] = errors[0]
        else:
            busy_p = [b for _, b, _ in got]
            res["value"] = sum(tokens * w.L / b for b in busy_p)
            res["cores"] = procs
            res["sample"] = (f"{procs} processes at once, each replaying stream 0's tokens 0..{tokens - 1} "
                             f"through all {w.L} layers; {max(busy_p):.1f} s of oracle time per process")
    return res


def topk_near_ties(z, K):
    """Top-K boundary of the native logits z [L][S][N] (fp32, the last timed
    token): how many (layer, stream) pairs have their K-th and (K+1)-th
    largest logits equal, or one fp32 ulp apart, where a one-ulp difference
    from the fp64 sum could decide the selection."""
    import numpy as np
    pairs = z.shape[0] * z.shape[1]
    if K >= z.shape[-1]:
        return {"pairs": pairs, "equal": 0, "within_one_ulp": 0}
    zs = -np.sort(-z.astype(np.float32), axis=-1)
    kth, nxt = zs[..., K - 1], zs[..., K]
    gap = kth - nxt
    return {"pairs": pairs, "equal": int(np.sum(gap == 0)),
            "within_one_ulp": int(np.sum(gap <= np.spacing(np.abs(kth))))}


def paper_context(w):
    """The paper's own hit-rate and traffic figures for the method and backbone
    this workload stands in for (Tables 1 and 3, Section 4.1 metrics), quoted
    as context only: they come from post-trained routers on real text in a
    trace-driven simulator, not from the random-init routers here."""
    import json as _json
    rows = _json.load(open(PAPER_METRICS))["rows"]
    model = "gptoss" if w.name.startswith("gptoss") else "qwen3"
    method = {(0, 0): "Temporal Router", (0, 1): "LRU", (0, 2): "LFU", (0, 3): "LRFU",
              (1, 0): "Spatio-Temporal Router"}.get((w.mode, w.policy))
    table1 = [r for r in rows if r["model"] == model and r["method"] == method and r.get("capacity") is None]
    out = {
        "note": "context only: post-trained routers on GSM8K/MATH/CSQA in a trace-driven simulator; the "
                "synthetic workloads here use random-init routers, so the rates are not comparable",
        "hardware": "an eight-accelerator node with 140 GB of device memory per accelerator (Section 4.1); "
                    "the accelerator is not named",
        "precision": "bf16 experts (S_exp = 3 d F x 2 bytes reproduces every printed Load)",
        "main_settings": {"qwen3": "capacity 20, R 15", "gptoss": "capacity 8, R 6"}[model],
        "table1": [{k: r[k] for k in ("method", "task", "hit", "adj_hit", "load_mb")} for r in table1],
    }
    if w.zipf is not None:   # the capacity x refinement sweep stands in for Table 3
        out["table3"] = [{k: r[k] for k in ("method", "capacity", "R", "hit", "adj_hit", "load_mb")}
                         for r in rows if r.get("capacity") is not None]
    return out


def run_config(w, inputs, warmup, steps, profile_fill=False, fills=None):
    """One configuration through the C ABI: untimed warm-up tokens, then
    `steps` timed tokens.  Returns (seconds per token, stats, fill ms, fill
    launches)."""
    import torch

    from paper_2609_04895_amd.workload import engine_for
    eng = engine_for(w, inputs, warmup_tokens=warmup, fills=fills)
    hidden = inputs["hidden"]
    y = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device="cuda:0")
    for t in range(warmup):
        eng.cmoe_step(hidden[t], y)
    torch.cuda.synchronize()
    if profile_fill:
        eng.cmoe_profile_begin(steps, kernels=("fill",))
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(eng.main_stream)
    for t in range(warmup, warmup + steps):
        eng.cmoe_step(hidden[t], y)
    ev1.record(eng.main_stream)
    torch.cuda.synchronize()
    sec = ev0.elapsed_time(ev1) / 1e3 / steps
    prof = eng.cmoe_profile_end() if profile_fill else None
    tot, _, _ = eng.cmoe_stats()
    eng.cmoe_destroy()
    fill_ms, fill_n = prof["fill"] if prof else (0.0, 0)
    return sec, tot, fill_ms, fill_n


def overlap_study(w, warmup, steps):
    """Exposed expert-loading time per decode token against Appendix B.3's
    fixed-trace model t_load(eta) = c_exp / T [D + (1 - eta) P], on one stream
    whose every logical load is a physical copy from the cold pool.

    Configurations on the same inputs: A = the workload (full mode, demand and
    proactive loads; proactive copies on the side stream overlap the previous
    layer's FFN), A_main = the same with the proactive copies in the demand
    fill launch on the main stream (no overlap), B = update-only (demand loads only, all on the critical
    path), Z = capacity N (after warm-up nearly every expert stays resident:
    the compute time of the same decode).  c_exp, the time of one expert copy,
    and the launch cost of a fill with nothing to copy, solve fill time =
    launches x t0 + copies x c_exp over the fill kernel's HIP events in B and Z.  The exposed load of a configuration is its time per
    token minus Z's, corrected for Z's few remaining copies."""
    import synth
    T = warmup + steps
    inputs = synth.device_inputs(w, T=T)
    cfgA = w
    cfgB = w.replace(mode=synth.MODE_TEMPORAL, R=0)
    cfgZ = w.replace(mode=synth.MODE_TEMPORAL, R=0, C=w.N)
    res = {}
    for name, cw, prof, fills in (("A", cfgA, False, "side"), ("A_main", cfgA, False, "main"), ("B", cfgB, False, None),
                                  ("B_fill_events", cfgB, True, None), ("Z", cfgZ, False, None),
                                  ("Z_fill_events", cfgZ, True, None)):
        sec, tot, fill_ms, fill_n = run_config(cw, inputs, warmup, steps, profile_fill=prof, fills=fills)
        A_, D_, P_, Tc = tot["accesses"], tot["demand_misses"], tot["proactive_loads"], tot["tokens"]
        res[name] = {"ms_per_token": sec * 1e3, "A": A_, "D": D_, "P": P_, "T": Tc,
                     "phys_fills": tot["phys_fills"], "hit": 1 - D_ / A_, "adj_hit": (A_ - D_) / (A_ + P_),
                     "load_mb_per_token": (D_ + P_) * w.expert_bytes / 1e6 / Tc,
                     "fill_ms": fill_ms, "fill_launches": fill_n}
        print(f"[overlap] {name}: {res[name]}", file=sys.stderr, flush=True)
    B, Bf, Z, Zf = res["B"], res["B_fill_events"], res["Z"], res["Z_fill_events"]
    # fill time = launches x t0 + copies x c_exp, from the two event runs
    nB, FB, nZ, FZ = Bf["fill_launches"], Bf["phys_fills"], Zf["fill_launches"], Zf["phys_fills"]
    c_exp = (Bf["fill_ms"] - Zf["fill_ms"] * nB / nZ) / (FB - FZ * nB / nZ)
    t0 = (Zf["fill_ms"] - FZ * c_exp) / nZ
    # Z still copies a few first-time experts; charge them at c_exp
    compute = Z["ms_per_token"] - Z["phys_fills"] * c_exp / Z["T"]
    out = {"study": "transfer overlap (Appendix B.3)", "workload": describe(w), "warmup": warmup, "steps": steps,
           "expert_bytes": w.expert_bytes, "c_exp_ms": c_exp, "copy_GBs": w.expert_bytes / (c_exp / 1e3) / 1e9,
           "empty_fill_launch_ms": t0, "compute_ms_per_token": compute, "configs": res}
    for name in ("A", "A_main", "B"):
        r = res[name]
        exposed = r["ms_per_token"] - compute
        lo_, hi_ = r["D"] * c_exp / r["T"], (r["D"] + r["P"]) * c_exp / r["T"]
        eta = 1.0 - (exposed - lo_) / (hi_ - lo_) if r["P"] > 0 else None
        out[name] = {"exposed_ms_per_token": exposed, "t_load_eta1_ms": lo_, "t_load_eta0_ms": hi_,
                     "eta_implied": eta}
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed decode tokens (default: T - warmup)")
    ap.add_argument("--warmup", type=int, default=16, help="untimed decode tokens before the timed region")
    ap.add_argument("--workload", default="qwen3_30b")
    ap.add_argument("--C", type=int, default=None)
    ap.add_argument("--R", type=int, default=None)
    ap.add_argument("--policy", choices=sorted(POLICIES), default=None,
                    help="retention priority (default: the workload's, the Temporal Router)")
    ap.add_argument("--mode", choices=sorted(MODES), default=None, help="default: the workload's mode")
    ap.add_argument("--lrfu-lambda", type=float, default=None)
    ap.add_argument("--layers", type=int, default=None, help="run the first L layers only")
    ap.add_argument("--streams", type=int, default=None, help="number of decode streams S (default: the workload's)")
    ap.add_argument("--arena-slots", type=int, default=None,
                    help="HBM expert slots per layer (default 0: min(N, S C), which holds the union of the caches)")
    ap.add_argument("--fills", choices=["auto", "main", "side"], default="auto",
                    help="where proactive fills run (auto: the library's choice, one launch with the demand fill "
                         "on the main stream)")
    ap.add_argument("--ffn-shape", choices=["auto", "single", "grouped"], default="auto",
                    help="bf16 FFN workgroups: one wavefront each, or four sharing big units' activations "
                         "(auto: the library's choice from the average tokens per expert)")
    ap.add_argument("--no-profile", action="store_true",
                    help="skip the second, event-timed pass (no roofline of the dominant kernel)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle time budget (0: skip)")
    ap.add_argument("--overlap-study", action="store_true",
                    help="instead of the benchmark line: measure exposed expert-loading time per token and the "
                         "transfer-overlap model of Appendix B.3 (use with --workload qwen3_30b_s1)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="after the timed region, run one elementwise device copy of 1 GiB (reference "
                         "kernel for scaling rocprofv3 byte counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the path shards by stream "
              "with no exchange, so the multi-GPU figure is not measured here", file=sys.stderr)
        sys.exit(2)

    import synth

    w = synth.WORKLOADS[args.workload]
    if args.C is not None or args.R is not None:
        w = w.replace(C=w.C if args.C is None else args.C, R=w.R if args.R is None else args.R)
    if args.policy is not None:
        w = w.replace(policy=POLICIES[args.policy])
    if args.mode is not None:
        w = w.replace(mode=MODES[args.mode])
    if args.lrfu_lambda is not None:
        w = w.replace(lrfu_lambda=args.lrfu_lambda)
    if args.layers is not None:
        w = w.replace(L=args.layers)
    if args.streams is not None:
        w = w.replace(S=args.streams)
    if args.arena_slots is not None:
        w = w.replace(arena_slots=args.arena_slots)
    warmup = args.warmup
    steps = args.steps if args.steps is not None else max(1, w.T - warmup)
    if args.overlap_study:
        print(json.dumps(overlap_study(w, warmup, min(steps, w.T - warmup))), flush=True)
        return

    # the oracle's leg forks worker processes: it runs before anything here
    # touches the GPU
    cb = None
    if args.cpu_seconds > 0:
        t0 = time.time()
        cb = cpu_baseline(w, args.cpu_seconds)
        # the whole workload (S streams x T tokens x L layers) at the sampled
        # rates: an extrapolation, not a measurement
        full = w.S * w.T * w.L
        cb["extrapolated_full_workload_s"] = {"one_core": full / cb["single_core"]["value"]}
        if cb["cores"] > 1:
            cb["extrapolated_full_workload_s"][f"{cb['cores']}_cores"] = full / cb["value"]
        print(f"[bench] oracle baseline done in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)

    import torch

    from paper_2609_04895_amd import cmoe as B
    from paper_2609_04895_amd.workload import engine_for

    # the second (event-timed) pass runs the tokens after the timed ones
    passes = 1 if args.no_profile else 2
    T_gen = min(w.T, warmup + passes * steps)
    print(f"[bench] {describe(w)}; warmup {warmup}, timed {steps}", file=sys.stderr, flush=True)

    t0 = time.time()
    inputs = synth.device_inputs(w, T=T_gen)
    print(f"[bench] inputs generated on the device in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    eng = engine_for(w, inputs, warmup_tokens=warmup, fills=args.fills, ffn_shape=args.ffn_shape)
    hidden = inputs["hidden"]
    y = torch.empty((w.S, w.L, w.d), dtype=torch.float32, device="cuda:0")
    main_stream = eng.main_stream

    for t in range(warmup):
        eng.cmoe_step(hidden[t % T_gen], y)
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(main_stream)
    for t in range(warmup, warmup + steps):
        eng.cmoe_step(hidden[t % T_gen], y)
    ev1.record(main_stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    elapsed = ev0.elapsed_time(ev1) / 1e3
    tot, _, _ = eng.cmoe_stats()
    active = eng.cmoe_read(B.CMOE_VIEW_ACTIVE)
    near_ties = topk_near_ties(eng.cmoe_read(B.CMOE_VIEW_LOGITS)[:, :, 0], w.K)
    print(f"[bench] timed region {elapsed * 1e3:.1f} ms (wall {wall * 1e3:.1f} ms)", file=sys.stderr, flush=True)

    e = w.elem_bytes
    n_act = int(active.sum())                 # expert weight reads by the FFN over the timed region
    launches = w.L * steps
    value = w.S * w.L * steps / elapsed
    res = {
        "metric": METRIC,
        "value": value,
        "unit": "token-layer steps/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": elapsed / steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == 1 else "f32",
        "data": "synthetic",
        "config": {"workload": describe(w), "streams": w.S, "layers": w.L, "experts": w.N, "top_k": w.K,
                   "capacity": w.C, "refine_budget": w.R if w.has_spatio else 0,
                   "mode": {0: "update-only", 1: "spatio-temporal", 2: "spatio-only"}[w.mode],
                   "retention": {v: k for k, v in POLICIES.items()}[w.policy], "d": w.d, "F": w.F,
                   "proactive_fills": fills_label(w, args.fills), "ffn_shape": args.ffn_shape,
                   "arena_slots": w.arena_slots or min(w.N, w.S * w.C)},
    }
    # algorithmic bytes of one token step: each distinct selected expert read
    # once, router weights, hidden states in, layer outputs out, fills (read +
    # write of each copied expert)
    step_bytes = (n_act * w.expert_bytes + steps * w.L * (w.n_routers * w.N * w.d * e + w.S * w.d * e
                                                          + w.S * w.d * 4)
                  + 2 * tot["phys_bytes"]) / steps
    res["step_hbm"] = {"algorithmic_bytes": step_bytes, "achieved_GBs": step_bytes / (elapsed / steps) / 1e9,
                       "frac": step_bytes / (elapsed / steps) / 1e9 / HBM_PEAK_GBS}
    if w.pool_kind == synth.POOL_HOST_PINNED:
        # expert copies out of the pinned host pool cross the host link
        res["host_link"] = {"copied_bytes_per_step": tot["phys_bytes"] / steps,
                            "achieved_GBs": tot["phys_bytes"] / elapsed / 1e9}
    if passes == 2:
        # the same number of tokens again, each gate/up launch carrying a HIP
        # event pair that takes the kernel's own start and end timestamps
        eng.cmoe_profile_begin(steps, kernels=("ffn_up",))
        p0 = torch.cuda.Event(enable_timing=True)
        p1 = torch.cuda.Event(enable_timing=True)
        p0.record(main_stream)
        for t in range(warmup + steps, warmup + 2 * steps):
            eng.cmoe_step(hidden[t % T_gen], y)
        p1.record(main_stream)
        torch.cuda.synchronize()
        prof = eng.cmoe_profile_end()
        n_act_p = int(eng.cmoe_read(B.CMOE_VIEW_ACTIVE).sum()) - n_act
        ms_up, n_up = prof["ffn_up"]
        avg_s = ms_up / 1e3 / max(n_up, 1)
        bytes_up = (n_act_p * 2 * w.F * w.d * e) / (w.L * steps) + w.S * w.d * e + w.S * w.K * w.F * e
        gbs = bytes_up / avg_s / 1e9
        res["roofline"] = {"kernel": "ffn_up_bf16" if w.dtype == 1 else "ffn_up_f32", "bound": "hbm",
                           "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                           "traffic": measured_traffic(w), "avg_launch_us": avg_s * 1e6,
                           "algorithmic_bytes_per_launch": bytes_up,
                           "timed_by": f"HIP events on each of its {n_up} launches in a second pass of {steps} "
                                       f"tokens after the timed region",
                           "second_pass_ms_per_step": p0.elapsed_time(p1) / steps}

    A, D, P, Tc = tot["accesses"], tot["demand_misses"], tot["proactive_loads"], tot["tokens"]
    res["cache"] = {"hit": 1 - D / A, "adj_hit": (A - D) / (A + P), "load_mb_per_token": (D + P) * w.expert_bytes
                    / 1e6 / Tc, "accesses": A, "demand_misses": D, "proactive_loads": P, "tokens": Tc,
                    "phys_fills": tot["phys_fills"], "distinct_experts_per_layer_step": n_act / launches,
                    "topk_near_ties_last_token": near_ties}
    eff, ent, fmax, top8 = eng.cmoe_concentration(8)
    res["concentration"] = {"effective_experts": eff, "entropy_nats": ent, "max_frequency": fmax, "top8_mass": top8}
    res["paper_context"] = paper_context(w)
    print(f"[bench] {json.dumps(res)}", file=sys.stderr, flush=True)
    eng.cmoe_destroy()
    del inputs, hidden
    if "roofline" in res:
        # second reference: a plain 1 GiB device copy in the same process
        # (bytes read + bytes written per second)
        src = torch.empty(1 << 28, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(5):
            dst.copy_(src)
        c1.record()
        torch.cuda.synchronize()
        copy_gbs = 5 * 2 * (1 << 30) / (c0.elapsed_time(c1) / 1e3) / 1e9
        res["roofline"]["device_copy_GBs"] = copy_gbs
        res["roofline"]["frac_of_device_copy"] = res["roofline"]["achieved"] / copy_gbs
        # third reference: the practical ceiling of a weight stream, a 1 GiB
        # read with the FFN's load pattern (cmoe_read_probe), best of 5
        ceil_gbs = B.cmoe_read_probe(src.view(torch.uint8), reps=5)
        res["roofline"]["read_ceiling_GBs"] = ceil_gbs
        res["roofline"]["frac_of_read_ceiling"] = res["roofline"]["achieved"] / ceil_gbs
        del src, dst
    if args.calibrate_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")   # 1 GiB
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)   # one elementwise kernel: reads 1 GiB, writes 1 GiB
        torch.cuda.synchronize()
        del src, dst
    if cb is not None:
        res["cpu_baseline"] = cb
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
