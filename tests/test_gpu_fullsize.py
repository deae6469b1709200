"""GPU vs oracle at the benchmark workloads' full sizes (B environments), in the launch
shapes bench.py times: av_step_n launches of 1000 steps (the workload benchmarks), of 20
steps (the default line's timed launches) and one-step av_step launches.

Environments are independent, so the oracle steps a sample of them (first, last, both halves
of lane words, random others) over every step.  Rewards and done flags are compared at every
step; the sampled maps are compared after every launch.  The first launch is 37 steps long, so
launch ends fall on steps 1000 k + 37: never on a multiple of the episode length (100), where
an environment whose episode did not end early would just have been reset to its initial map.
Every config x variant runs (15 pairs), on the engine AUTO picks for it (the per-environment
rule sets of c2 and c3 on the group engine, at the occupancy their full batch sizes set)."""
import numpy as np
import pytest

import oracle
from gpu_util import require_gpu, say
import paper_2407_04221_amd as av
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu

CASES = [(n, v) for n in ("c1", "c2", "c3", "c4", "c5") for v in ("literal", "planted", "dense")]
OFFSET = 37


def sample_envs(B, k, seed):
    g = np.random.default_rng(seed)
    fixed = [0, 1, B - 2, B - 1, B // 2, B // 2 + 1]
    rest = g.choice(B, size=min(B, k), replace=False).tolist()
    return sorted(set(e for e in fixed + rest if 0 <= e < B))


def launch_plan(T, chunk):
    """Launch lengths: OFFSET first, then chunk-step launches up to T + OFFSET steps."""
    plan, t = [min(OFFSET, T + OFFSET)], OFFSET
    while t < T + OFFSET:
        k = min(chunk, T + OFFSET - t)
        plan.append(k)
        t += k
    return plan


def run_sampled(wl, maps, rules, actions, plan, envs, api="step_n"):
    """GPU run of the whole batch in the launch lengths of `plan`; returns rewards / done
    [T][B] and the sampled environments' maps after each launch ([launches][n][C][H][W])."""
    import torch
    T = int(sum(plan))
    b = av.Batch.for_workload(wl)
    idx = torch.as_tensor(envs, device="cuda")
    try:
        b.load_rules(*rules)
        b.reset(maps)
        acts = torch.from_numpy(np.ascontiguousarray(actions[:T])).cuda()
        rew = torch.empty((T, wl.B), dtype=torch.float32, device="cuda")
        don = torch.empty((T, wl.B), dtype=torch.uint8, device="cuda")
        full = torch.empty((wl.B, wl.C, wl.H, wl.W), dtype=torch.uint8, device="cuda")
        snaps = []
        t = 0
        for k in plan:
            if api == "step":
                for u in range(t, t + k):
                    av.av_step(b.h, acts[u], rew[u], don[u])
            else:
                av.av_step_n(b.h, k, acts[t:t + k], rew[t:t + k], don[t:t + k])
            t += k
            b.maps(out=full)
            snaps.append(full.index_select(0, idx).cpu().numpy())
        eng = av.ENGINE_NAMES[b.info["engine"]]
        return rew.cpu().numpy(), don.cpu().numpy(), np.stack(snaps), eng
    finally:
        b.close()


def oracle_sampled(wl, maps, rules, actions, plan, envs):
    """The oracle on the sampled environments: rewards / done [T][n] and maps after every
    launch of `plan`."""
    m_s, r_s, a_s = inputs.subset_envs(wl, maps, rules, actions, envs)
    o = oracle.Oracle.for_workload(wl, B=len(envs))
    try:
        o.load_rules(*r_s)
        o.reset(m_s)
        T = int(sum(plan))
        rew = np.zeros((T, len(envs)), np.float32)
        don = np.zeros((T, len(envs)), np.uint8)
        snaps = []
        t = 0
        for k in plan:
            for u in range(t, t + k):
                rew[u], don[u] = o.step(a_s[u], 8)
            t += k
            snaps.append(o.maps())
        return rew, don, np.stack(snaps)
    finally:
        o.close()


def check(wl, variant, plan, envs, got, want):
    r, d, snaps, eng = got
    wr, wd, wsnaps = want
    for li, t_end in enumerate(np.cumsum(plan)):
        t0 = t_end - plan[li]
        np.testing.assert_array_equal(r[t0:t_end][:, envs], wr[t0:t_end],
                                      err_msg=f"rewards, launch {li} (steps {t0}..{t_end - 1})")
        np.testing.assert_array_equal(d[t0:t_end][:, envs], wd[t0:t_end],
                                      err_msg=f"done, launch {li} (steps {t0}..{t_end - 1})")
        np.testing.assert_array_equal(snaps[li], wsnaps[li],
                                      err_msg=f"maps after launch {li} (step {t_end - 1})")
    # not vacuous: episodes end early or by length, the sampled maps are not their initial
    # maps at the launch ends, and (except literal rules) rewards are paid
    assert wd.any()
    return eng


@pytest.mark.parametrize("name,variant", CASES, ids=[f"{n}-{v}" for n, v in CASES])
def test_full_size_bench_launches(name, variant):
    require_gpu()
    wl = inputs.WORKLOADS[name]
    plan = launch_plan(wl.T, 1000)
    say(f"[fullsize] {name} {variant}: B={wl.B} launches {plan}")
    maps, rules, actions = inputs.make_all(wl, 0, variant, T=int(sum(plan)))
    envs = sample_envs(wl.B, 10 if name in ("c3", "c5") else 16, seed=wl.config_id)
    got = run_sampled(wl, maps, rules, actions, plan, envs)
    say(f"[fullsize] {name} {variant}: GPU done (engine {got[3]}); oracle on {len(envs)} envs")
    want = oracle_sampled(wl, maps, rules, actions, plan, envs)
    check(wl, variant, plan, envs, got, want)
    init = maps[envs]
    moved = [not np.array_equal(s, init) for s in want[2]]
    assert all(moved), "a launch ended with every sampled map equal to its initial map"
    if variant != "literal" and (name, variant) != ("c5", "dense"):
        # loaded rules fired: rewards were paid, or (c5's shared planted set fires once, in
        # environment 0 at t = 0, with rewards that sum to zero) some map holds more than one
        # player cell, which no move can make.  c5's dense set does not fire: its 5 x 5 rules
        # over 13 channels keep about 32 specified entries each, which random maps never meet.
        players = want[2][:, :, 2].sum(axis=(-1, -2))
        assert (want[0] != 0).any() or (players > 1).any()
    # properties of every environment, not just the sample
    r, d = got[0], got[1]
    assert d.max() <= 1 and np.array_equal(r, np.round(r))
    expect = {"c1": "lane16", "c2": "group", "c3": "group", "c4": "lane16", "c5": "rows"}
    assert got[3] == expect[name]


def test_full_size_default_line_launches():
    """c4 in the default bench line's shapes: 20-step av_step_n launches and one-step av_step
    launches, sampled maps after every launch."""
    require_gpu()
    wl = inputs.WORKLOADS["c4"]
    for api, chunk, steps in (("step_n", 20, 263), ("step", 1, 137)):
        plan = launch_plan(steps, chunk)
        say(f"[fullsize default] c4 {api}: {len(plan)} launches")
        maps, rules, actions = inputs.make_all(wl, 1, "planted", T=int(sum(plan)))
        envs = sample_envs(wl.B, 16, seed=41)
        got = run_sampled(wl, maps, rules, actions, plan, envs, api=api)
        want = oracle_sampled(wl, maps, rules, actions, plan, envs)
        check(wl, "planted", plan, envs, got, want)


def test_quarter_million_environments_sampled():
    """A batch 16 times the throughput workload's (262144 environments of c4's shape) in
    1000-step launches: grid indexing past the workload's size, sampled envs against the
    oracle over every step."""
    require_gpu()
    wl = inputs.WORKLOADS["c4"].with_(B=1 << 18, T=60, L=25)
    plan = launch_plan(wl.T, 1000)
    say(f"[fullsize] c4 x16: B={wl.B} launches {plan}")
    maps, rules, actions = inputs.make_all(wl, 3, "planted", T=int(sum(plan)))
    envs = sample_envs(wl.B, 24, seed=99)
    got = run_sampled(wl, maps, rules, actions, plan, envs)
    assert got[3] == "lane16"
    want = oracle_sampled(wl, maps, rules, actions, plan, envs)
    check(wl, "planted", plan, envs, got, want)
    assert (want[0] != 0).any()
