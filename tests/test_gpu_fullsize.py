"""GPU vs oracle at the benchmark workloads' full sizes (B environments, T steps), in the
launch shape bench.py times (av_step_n launches of 1000 steps).  Environments are
independent, so the oracle steps a sample of them (first, last, both halves of lane words,
random others) over all T steps; rewards and done flags are compared at every step and the
maps after the last step."""
import numpy as np
import pytest

import oracle
from gpu_util import gpu_run, require_gpu, say
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu

CASES = [("c1", "literal"), ("c1", "dense"), ("c2", "literal"), ("c2", "dense"),
         ("c3", "literal"), ("c4", "literal"), ("c4", "planted"), ("c4", "dense"),
         ("c5", "literal")]


def sample_envs(B, k, seed):
    g = np.random.default_rng(seed)
    fixed = [0, 1, B - 2, B - 1, B // 2, B // 2 + 1]
    rest = g.choice(B, size=min(B, k), replace=False).tolist()
    return sorted(set(e for e in fixed + rest if 0 <= e < B))


@pytest.mark.parametrize("name,variant", CASES, ids=[f"{n}-{v}" for n, v in CASES])
def test_full_size_sampled(name, variant):
    require_gpu()
    wl = inputs.WORKLOADS[name]
    say(f"[fullsize] {name} {variant}: B={wl.B} T={wl.T}")
    maps, rules, actions = inputs.make_all(wl, 0, variant)
    _, final, r, d, eng = gpu_run(wl, maps, rules, actions, mode="step_n", chunk=1000)
    say(f"[fullsize] {name} {variant}: GPU done (engine {eng}); oracle on a sample")
    envs = sample_envs(wl.B, 10 if name in ("c3", "c5") else 16, seed=wl.config_id)
    m_s, r_s, a_s = inputs.subset_envs(wl, maps, rules, actions, envs)
    want_m, want_r, want_d = oracle.run(wl, m_s, r_s, a_s, nthreads=8)
    np.testing.assert_array_equal(r[:, envs], want_r, err_msg="rewards")
    np.testing.assert_array_equal(d[:, envs], want_d, err_msg="done")
    np.testing.assert_array_equal(final[envs], want_m[-1], err_msg="final maps")
    # the run is not trivial: episodes end, and (except literal rules) rewards are paid
    assert want_d.any()
    if variant != "literal":
        assert (want_r != 0).any()
    # properties that hold for every environment, not just the sample
    assert set(np.unique(final)) <= {0, 1}
    assert d.max() <= 1
    assert np.array_equal(r, np.round(r))


def test_quarter_million_environments_sampled():
    """A batch 16 times the throughput workload's (262144 environments of c4's shape) in the
    launch shape bench.py times: grid indexing past the workload's size, sampled envs against
    the oracle over every step."""
    require_gpu()
    wl = inputs.WORKLOADS["c4"].with_(B=1 << 18, T=60, L=25)
    say(f"[fullsize] c4 x16: B={wl.B} T={wl.T}")
    maps, rules, actions = inputs.make_all(wl, 3, "planted")
    _, final, r, d, eng = gpu_run(wl, maps, rules, actions, mode="step_n", chunk=1000)
    assert eng == 2                         # lane16
    envs = sample_envs(wl.B, 24, seed=99)
    m_s, r_s, a_s = inputs.subset_envs(wl, maps, rules, actions, envs)
    want_m, want_r, want_d = oracle.run(wl, m_s, r_s, a_s, nthreads=8)
    np.testing.assert_array_equal(r[:, envs], want_r, err_msg="rewards")
    np.testing.assert_array_equal(d[:, envs], want_d, err_msg="done")
    np.testing.assert_array_equal(final[envs], want_m[-1], err_msg="final maps")
    assert want_d.any() and (want_r != 0).any()
