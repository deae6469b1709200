"""Benchmark of the batched rule step on one MI355X.

Default workload: 16384 environments, 16x16 maps, 6 channels, 8 shared 3x3 rules (30 %
don't-care entries), random actions, episodes of 100 steps, 5000 steps: the throughput
workload.  Prints one JSON line with env-steps/s (whole batch), cell-rule-updates/s, the
fraction of the HBM roofline for the step kernel, and the CPU oracle's rate on a bounded
sample of the same workload on this host.

Timing: `--steps` steps in av_step_n launches of up to `--chunk` steps, repeated (at least
five times) after `--warmup` untimed steps; each repeat is bracketed by HIP events on the
launch stream, and the median is reported with every repeat listed.

Roofline of the multi-step launch: VALU-bound (the maps stay on chip between its steps), so
`roofline` is VALU lane-ops per launch (from committed counters of the same launch shape) over
the launch's duration against 256 CUs x 64 lanes x 2.4 GHz.  The workload metric's HBM
normaliser, A = 2*C*H*W/8 (packed maps in and out) + 6 (action u8, reward f32, done u8) bytes
per env-step at 8 TB/s, is reported beside it and for the one-launch-per-step path
(`per_launch_path`), which does move A bytes per env-step.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "env-steps/sec and cell-rule-updates/sec at 1 MI355X; % of HBM roofline"
# the sources that determine each engine's step kernel (the lane16 body is generated)
KERNEL_SOURCES = {
    "generic": ("paper_2407_04221_amd/csrc/k_generic.hip",),
    "wave": ("paper_2407_04221_amd/csrc/k_wave.hip",),
    "rows": ("paper_2407_04221_amd/csrc/k_rows.hip",),
    "group": ("paper_2407_04221_amd/csrc/k_group.hip",),
    "lane16": ("paper_2407_04221_amd/csrc/lane16_kernel.hip",
               "paper_2407_04221_amd/csrc/lane16_jit.cpp",
               "paper_2407_04221_amd/csrc/codegen.h"),
}


def kernel_hash(engine: str) -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[engine]:
        p = os.path.join(ROOT, rel)
        if os.path.exists(p):
            h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def algorithmic_bytes(wl) -> int:
    return 2 * wl.C * wl.H * wl.W // 8 + 6


def counter_record(key: str, engine_name: str):
    """Per-launch hardware counters of one launch shape (`workload/engine/variant/k=steps per
    launch`) from the committed rocprofv3 summaries, if they were taken on the current sources
    of that engine's kernel; otherwise None."""
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(key)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("kernel_hash") != kernel_hash(engine_name):
        return None
    return rec


def host_cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, maps, rules, actions, budget_s: float, threads: int,
                 rule_mode: str = "parallel", control=None):
    """The oracle as it stands on a bounded sample of the workload (the first 4096
    environments, as many steps as fit in budget_s; a workload of fewer steps than that is run
    again from its initial maps), OpenMP over environments on `threads` host threads, then
    single-threaded for a quarter of the budget."""
    import oracle
    from paper_2407_04221_amd import inputs
    nb = min(wl.B, 4096)
    envs = np.arange(nb)
    m, r, a = inputs.subset_envs(wl, maps, rules, actions, envs)

    def timed(nthreads, budget):
        o = oracle.Oracle.for_workload(wl, B=nb, rule_mode=int(rule_mode == "sequential"))
        o.load_rules(*r)
        if control is not None:
            limit, inhibit, order, seed = control
            S = nb if wl.per_env else 1
            o.set_rule_control(limit[:S], inhibit[:S], order, seed)
        o.reset(m)
        steps = 0
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < budget:
            if steps and steps % a.shape[0] == 0:
                o.reset(m)                        # another pass over the workload's steps
            o.step(a[steps % a.shape[0]], nthreads=nthreads)
            steps += 1
        dt = time.perf_counter() - t0
        used = o.threads_used
        o.close()
        return nb * steps / dt, steps, dt, used

    value, steps, dt, used = timed(threads, budget_s)
    v1, s1, dt1, _ = timed(1, budget_s / 4)
    T = a.shape[0]

    def passes(n):
        return f" in {-(-n // T)} passes of {T}" if n > T else ""

    return {"value": value, "unit": "env-steps/s", "cores": used, "kind": "oracle",
            "sample": f"first {nb} of {wl.B} envs x {steps} steps{passes(steps)} ({dt:.1f} s, "
                      f"{used} threads of {os.cpu_count()} on {host_cpu_model()})",
            "single_thread": {"value": v1,
                              "sample": f"first {nb} envs x {s1} steps{passes(s1)} ({dt1:.1f} s)"}}


def _time_us(fn, stream, torch, reps=100):
    fn()
    torch.cuda.synchronize()
    g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g0.record(stream)
    for _ in range(reps):
        fn()
    g1.record(stream)
    torch.cuda.synchronize()
    return g0.elapsed_time(g1) * 1e3 / reps


def bench_mutation(av, torch, wl, maps, rules, stream, seed):
    """av_mutate_maps over the population's initial maps (uint8, read + written once) and
    av_mutate_rules over its rule arrays; HBM bytes are the arrays read and written."""
    m = av.mutation(seed=seed, generation=1, map_flip=0.01, entry=0.05, reward=0.1)
    src = torch.from_numpy(maps).cuda()
    dst = torch.empty_like(src)
    us_maps = _time_us(lambda: av.av_mutate_maps(src, dst, m), stream, torch)
    map_bytes = 2 * maps.size
    dev = [torch.from_numpy(np.ascontiguousarray(x)).cuda() for x in rules]
    out = [torch.empty_like(x) for x in dev[1:]]
    us_rules = _time_us(lambda: av.av_mutate_rules(*dev, *out, m), stream, torch)
    rule_bytes = (2 * (rules[1].size + rules[2].size) + 2 * 4 * rules[3].size
                  + 4 * rules[0].size)

    def roof(nbytes, us):
        gbs = nbytes / (us * 1e-6) / 1e9
        return {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": gbs / HBM_PEAK_GBS, "bytes_per_call": int(nbytes)}

    return {"maps": {"api": "av_mutate_maps", "individuals": int(maps.shape[0]),
                     "us_per_call": us_maps, "individuals_per_sec": maps.shape[0] / (us_maps * 1e-6),
                     "philox_blocks_per_call": int(maps.shape[0] * ((maps[0].size + 7) // 8)),
                     "roofline": roof(map_bytes, us_maps)},
            "rules": {"api": "av_mutate_rules", "sets": int(rules[1].shape[0]),
                      "us_per_call": us_rules, "roofline": roof(rule_bytes, us_rules)}}


def bench_search(av, torch, wl, args):
    """av_search_* from environment 0's map and rule set: levels until the frontier empties or
    the budget of visits is spent.  Timed with the host clock around the whole search (each
    level synchronises once).  Bytes per visit: the packed state S = C x H x row bytes moved
    five times (gathered in, stepped in and out, hashed, copied to the frontier) plus 28 bytes
    of table slot and 20 of per-child metadata."""
    from paper_2407_04221_amd import inputs
    maps, rules, _ = inputs.make_all(wl, args.seed, args.search_variant, T=1)
    rules = tuple(x[:1] for x in rules)
    table_log2 = max(10, min(30, int(np.ceil(np.log2(max(2 * args.search, 16))))))
    g = av.Search(wl.H, wl.W, wl.C, wl.R, wl.max_h, wl.max_w, wl.L, num_actions=5,
                  max_frontier=args.search_frontier, table_log2=table_log2,
                  best_first_k=args.search_k, max_nodes=max(16, args.search + 1))
    g.load_rules(*rules)
    g.run(maps[0], min(args.search, 20000))          # warm-up (kernels, JIT)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    levels = g.run(maps[0], args.search)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    g.close()
    visited = levels[-1]["visited"] if levels else 0
    row_bytes = 2 if wl.W <= 16 else (4 if wl.W <= 32 else 8)
    S = wl.C * wl.H * row_bytes
    per_visit = 5 * S + 48
    gbs = visited * per_visit / dt / 1e9
    return {"api": "av_search_expand", "variant": args.search_variant, "budget": args.search,
            "order": f"best-first k={args.search_k}" if args.search_k else "level",
            "visited": visited, "levels": len(levels), "seconds": dt,
            "visits_per_sec": visited / dt, "best_reward": levels[-1]["best_reward"] if levels else 0,
            "best_visit": levels[-1]["best_visit"] if levels else 0,
            "frontier_peak": max((lv["frontier"] for lv in levels), default=0),
            "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": gbs / HBM_PEAK_GBS, "bytes_per_visit": per_visit},
            "level_sizes": [lv["children"] for lv in levels][:64]}


VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12   # 32-bit lane-ops/s: CUs x SIMDs x lanes x clock


def make_hold(torch):
    """A short device-side wait queued before a timed region: the launches of the region are
    queued behind it while it runs, so the region's start event fires with the work already
    queued and the events bracket device time, not the host's submission of the launches."""
    sleep = getattr(torch.cuda, "_sleep", None)
    if sleep is None:
        return None
    return lambda: sleep(2_000_000)


def timed_repeats(torch, stream, fn, repeats, hold):
    """Run fn() `repeats` times, each between two HIP events on `stream` (synchronised on both
    sides, a hold queued before the start event); returns the per-repeat times in ms."""
    out = []
    for _ in range(repeats):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if hold:
            hold()
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1))
    return out


def per_launch_path(av, torch, b, acts, n, repeats, hold, roof_env_steps, B):
    """One av_step launch per step for n steps: captured once in a HIP graph and replayed
    (device cost of a one-step launch), and called from Python (what a Python agent loop
    pays: ctypes marshalling and launch per step)."""
    rew = torch.empty((n, B), dtype=torch.float32, device="cuda")
    don = torch.empty((n, B), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(stream)
    try:
        with torch.cuda.stream(s):
            av.av_set_stream(b.h, s)
            with torch.cuda.graph(g, stream=s):
                for t in range(n):
                    av.av_step(b.h, acts[t % acts.shape[0]], rew[t], don[t])
    finally:
        stream.wait_stream(s)
        av.av_set_stream(b.h, stream)
    g.replay()
    graph_ms = timed_repeats(torch, stream, g.replay, repeats, hold)

    def eager():
        for t in range(n):
            av.av_step(b.h, acts[t % acts.shape[0]], rew[t], don[t])
    eager()
    py_ms = timed_repeats(torch, stream, eager, repeats, None)
    g_us = float(np.median(graph_ms)) * 1e3 / n
    p_us = float(np.median(py_ms)) * 1e3 / n
    return {"api": "av_step", "steps": n,
            "graph_us_per_step": g_us, "graph_repeats_ms": graph_ms,
            "graph_env_steps_per_sec": B / (g_us * 1e-6),
            "graph_frac_hbm_roofline": B / (g_us * 1e-6) / roof_env_steps,
            "python_us_per_step": p_us, "python_repeats_ms": py_ms,
            "python_frac_hbm_roofline": B / (p_us * 1e-6) / roof_env_steps,
            "note": "one launch per step moves A bytes per env-step through memory (maps in "
                    "and out, action, reward, done), so this path is measured against the HBM "
                    "roofline; graph: n launches captured once and replayed (device time, a "
                    "hold queued first); python: n av_step calls from Python per repeat"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: workload T)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps before timing (default: one launch of --chunk steps)")
    ap.add_argument("--repeats", type=int, default=7,
                    help="timed repeats of the --steps region; the median is reported")
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--variant", default="literal", choices=["literal", "planted", "dense"])
    ap.add_argument("--engine", default="auto",
                    choices=["auto", "generic", "lane16", "wave", "rows", "group"])
    ap.add_argument("--rule-mode", default="parallel", choices=["parallel", "sequential"])
    ap.add_argument("--limit", type=int, default=0,
                    help="rule application control: cap every loaded rule at K matches per step")
    ap.add_argument("--inhibit-chain", action="store_true",
                    help="rule application control: loaded rule r is inhibited by rule r - 1")
    ap.add_argument("--site-order", default="rowmajor", choices=["rowmajor", "random"])
    ap.add_argument("--chunk", type=int, default=1000, help="steps per av_step_n launch")
    ap.add_argument("--launch-steps", type=int, default=None,
                    help="steps of the one-launch-per-step path (av_step; default: --steps, at "
                         "most 100; 0 = skip)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="before timing, copy MIB MiB with a plain device copy (a known-size "
                         "reference for the HBM byte counters)")
    ap.add_argument("--observe", type=int, default=0, metavar="W",
                    help="also time av_observe with a W x W window (HBM-bound gather)")
    ap.add_argument("--mutate", action="store_true",
                    help="also time the mutation operators on the workload's population")
    ap.add_argument("--search", type=int, default=0, metavar="BUDGET",
                    help="also time the batched search from environment 0 with this many visits")
    ap.add_argument("--search-variant", default="dense", choices=["literal", "planted", "dense"])
    ap.add_argument("--search-frontier", type=int, default=1 << 20)
    ap.add_argument("--search-k", type=int, default=0,
                    help="batched best-first popping K nodes per iteration (0: level order)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU: the library has no multi-GPU path (asked for "
              f"--gpus {args.gpus}); environments are independent, so N GPUs would each run "
              f"this same kernel on B/N environments.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2407_04221_amd as av
    from paper_2407_04221_amd import inputs

    wl = inputs.WORKLOADS[args.workload]
    T = wl.T if args.steps is None else args.steps
    if args.warmup is None:
        args.warmup = min(args.chunk, T)
    repeats = max(5, args.repeats)
    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    maps, rules, actions = inputs.make_all(wl, args.seed, args.variant, T=max(T, args.warmup, 1))
    acts = torch.from_numpy(actions).cuda()
    b = av.Batch.for_workload(wl, engine=args.engine, rule_mode=args.rule_mode)
    b.load_rules(*rules)
    control = None
    if args.limit or args.inhibit_chain:
        S = wl.B if wl.per_env else 1
        limit = np.full((S, wl.R), args.limit, np.int32)
        inhibit = np.zeros((S, wl.R, wl.R), np.uint8)
        if args.inhibit_chain:
            for r in range(1, wl.R):
                inhibit[:, r - 1, r] = 1
        control = (limit, inhibit, av.SITE_ORDERS[args.site_order], args.seed)
        b.set_rule_control(*control)
    b.reset(maps)
    engine = b.info["engine"]
    engine_name = av.ENGINE_NAMES[engine]
    chunk = max(1, min(args.chunk, T))
    rew = torch.empty((chunk, wl.B), dtype=torch.float32, device="cuda")
    don = torch.empty((chunk, wl.B), dtype=torch.uint8, device="cuda")
    pos = [0]                                   # next action row (the actions repeat)

    def run(n_steps):
        launches = 0
        t = 0
        while t < n_steps:
            lo = pos[0] % actions.shape[0]
            k = min(chunk, n_steps - t, actions.shape[0] - lo)
            av.av_step_n(b.h, k, acts[lo:lo + k], rew[:k], don[:k])
            t += k
            pos[0] += k
            launches += 1
        return launches

    if args.warmup:
        run(args.warmup)
    b.reset(maps)
    pos[0] = 0
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    hold = make_hold(torch)
    launches = [0]

    def region():
        launches[0] = run(T)
    rep_ms = timed_repeats(torch, stream, region, repeats, hold)
    ms = float(np.median(rep_ms))
    # the same events around an empty region after the same hold: what the window costs with
    # no launch in it
    floor_us = float(np.median(timed_repeats(torch, stream, lambda: None, repeats, hold))) * 1e3

    # the kernel's average launch duration: `nb` launches of the timed shape back to back
    # between two events, so the events' own cost (event_floor_us for an empty window) is
    # spread over them; this is what a kernel trace reports per launch
    nb = max(3, min(50, 20000 // chunk))
    nl = [0]

    def back_to_back():
        nl[0] = run(nb * chunk)
    b2b_ms = float(np.median(timed_repeats(torch, stream, back_to_back, 3, hold)))
    launch_ms = b2b_ms / nl[0]

    env_steps = wl.B * T
    value = env_steps / (ms / 1e3)
    A = algorithmic_bytes(wl)
    roof_env_steps = HBM_PEAK_GBS * 1e9 / A
    steps_per_launch = T / launches[0]
    key = f"{args.workload}/{engine_name}/{args.variant}/k={chunk}"
    plain = control is None and args.rule_mode == "parallel" and args.seed == 0
    rec = counter_record(key, engine_name) if plain and T % chunk == 0 else None
    kernel = rec["kernel"] if rec else f"av_{engine_name}_step"
    valu_ops = rec["valu_insts_per_launch"] * 64 if rec else None
    achieved = valu_ops / (launch_ms * 1e-3) / 1e12 if valu_ops else None

    per_launch = None
    n1 = min(T, 100) if args.launch_steps is None else args.launch_steps
    if n1:
        b.reset(maps)
        torch.cuda.synchronize()
        per_launch = per_launch_path(av, torch, b, acts, n1, repeats, hold, roof_env_steps, wl.B)

    observe = None
    if args.observe:
        w = args.observe
        obs = torch.empty((wl.B, wl.C, w, w), dtype=torch.uint8, device="cuda")
        av.av_observe(b.h, w, obs)
        torch.cuda.synchronize()
        us = _time_us(lambda: av.av_observe(b.h, w, obs), stream, torch, reps=200)
        moved = wl.B * (wl.C * w * w + wl.C * wl.H * wl.W // 8)   # window out, packed maps in
        # one step and its observation per call, as an agent needs them: fused (the lane16
        # kernel writes the window from its registers) against a step then av_observe
        a1 = acts[:1]
        r1 = torch.empty((1, wl.B), dtype=torch.float32, device="cuda")
        d1 = torch.empty((1, wl.B), dtype=torch.uint8, device="cuda")
        us_fused = _time_us(lambda: av.av_step_observe(b.h, 1, a1, r1, d1, w, obs), stream, torch)

        def separate():
            av.av_step_n(b.h, 1, a1, r1, d1)
            av.av_observe(b.h, w, obs)
        us_sep = _time_us(separate, stream, torch)
        observe = {"api": "av_observe", "w": w, "us_per_call": us,
                   "step_observe_us": us_fused, "step_then_observe_us": us_sep,
                   "obs_per_sec": wl.B / (us * 1e-6),
                   "roofline": {"bound": "hbm", "achieved": moved / (us * 1e-6) / 1e9,
                                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                "frac": moved / (us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                                "bytes_per_call": moved}}

    search = None
    if args.search:
        search = bench_search(av, torch, wl, args)

    mutate = None
    if args.mutate:
        mutate = bench_mutation(av, torch, wl, maps, rules, stream, args.seed)

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(wl, maps, rules, actions, args.cpu_seconds,
                           threads=min(16, os.cpu_count() or 1), rule_mode=args.rule_mode,
                           control=control)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "env-steps/s",
        "n_gpus": 1,
        "steps": T,
        "warmup": args.warmup,
        "ms_per_step": ms / T,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: {wl.B} envs, {wl.H}x{wl.W} maps, C={wl.C}, R={wl.R} "
                        f"{'per-env' if wl.per_env else 'shared'} rules "
                        f"{'/'.join(f'{n}x{m}' for n, m in wl.shapes)}, p_dc={wl.p_dc:.2f}, "
                        f"{args.variant}, episode {wl.L} steps",
            "B": wl.B, "H": wl.H, "W": wl.W, "C": wl.C, "R": wl.R, "variant": args.variant,
            "engine": engine_name, "api": "av_step_n", "steps_per_launch": steps_per_launch,
            "launches_per_repeat": launches[0], "rule_mode": args.rule_mode,
            "control": None if control is None else {
                "limit": args.limit, "inhibit_chain": args.inhibit_chain,
                "site_order": args.site_order},
        },
        "repeats_ms": rep_ms,
        "event_floor_us": floor_us,
        # per step inside the kernel: the back-to-back launch duration (roofline.launch_ms) over
        # its steps, what a kernel trace of this launch shape shows; ms_per_step also holds the
        # event window's own cost, which is large against one short launch
        "kernel_ms_per_step": b2b_ms / (nb * chunk),
        "timing": "median of the repeats; each repeat times exactly `steps` steps between HIP "
                  "events on the launch stream, synchronised on both sides, with a device-side "
                  "hold queued before the start event so the launches are queued when it fires"
                  + ("" if hold else " (no hold available: host submission is inside the window)"),
        "cell_rule_updates_per_sec": value * wl.H * wl.W * wl.R,
        "roofline": {
            "bound": "alu", "achieved": achieved, "peak": VALU_PEAK_TOPS, "unit": "Tlane-op/s",
            "frac": None if achieved is None else achieved / VALU_PEAK_TOPS,
            "traffic": rec["bytes_per_launch"] if rec else None,
            "kernel": kernel, "launch_ms": launch_ms, "launches_back_to_back": nl[0],
            "valu_lane_ops_per_launch": valu_ops,
            "counters": rec["source"] if rec else None,
            "hbm_normaliser": {"algorithmic_bytes_per_env_step": A,
                               "achieved_gbs": A * value / 1e9,
                               "frac": A * value / 1e9 / HBM_PEAK_GBS},
            "note": "av_step_n keeps the maps on chip for the whole launch, so HBM carries only "
                    "actions, outputs and the maps once in and out (`traffic`); what bounds the "
                    "launch is VALU issue: achieved = VALU lane-ops per launch (SQ_INSTS_VALU x "
                    "64 from counters of this launch shape on these kernel sources) / the "
                    "launch's average duration (launch_ms: launches_back_to_back launches of "
                    "this shape between two events), against 256 CUs x 4 SIMDs x 16 lanes x "
                    "2.4 GHz; "
                    "hbm_normaliser is the workload metric's A bytes per env-step, which this "
                    "path does not move (one-launch-per-step: per_launch_path)",
        },
        "per_launch_path": per_launch,
        "observe": observe,
        "mutate": mutate,
        "search": search,
        "cpu_baseline": cpu,
    }
    b.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
