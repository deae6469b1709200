"""GPU path vs the CPU oracle, bit for bit, on the same seeded inputs.

Sizes here are ones the oracle finishes in seconds, with a ragged tail (B not a multiple
of the environments a workgroup or wave holds).  Maps, rewards and done flags are compared
after every step (av_step) or per step from av_step_n launches of ragged length."""
import numpy as np
import pytest

import oracle
from gpu_util import first_mismatch, gpu_run, group_ok, require_gpu, say
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu

# (workload, B, T): every benchmark workload, cut down in B and T
CASES = [("c1", 1, 100), ("c2", 203, 40), ("c3", 37, 30), ("c4", 333, 60), ("c5", 5, 20)]


def _case_ids():
    return [f"{n}-B{b}-T{t}" for n, b, t in CASES]


@pytest.mark.parametrize("variant", inputs.VARIANTS)
@pytest.mark.parametrize("seed", [0, 1])
@pytest.mark.parametrize("engine", ["generic", "wave", "rows", "group", "auto"])
@pytest.mark.parametrize("case", CASES, ids=_case_ids())
def test_step_matches_oracle(case, engine, seed, variant):
    require_gpu()
    name, B, T = case
    wl = inputs.WORKLOADS[name].with_(B=B, T=T, L=25)
    if engine == "group" and not group_ok(wl):
        pytest.skip("not eligible for the group engine")
    say(f"[parity] {name} B={B} T={T} engine={engine} seed={seed} variant={variant}")
    maps, rules, actions = inputs.make_all(wl, seed, variant)
    want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8)
    seq, final, r, d, eng = gpu_run(wl, maps, rules, actions, engine=engine, mode="step")
    for t in range(T):
        assert first_mismatch(seq[t], want_m[t]) is None, \
            f"maps differ at step {t}, index {first_mismatch(seq[t], want_m[t])}"
        assert first_mismatch(r[t], want_r[t]) is None, f"rewards differ at step {t}"
        assert first_mismatch(d[t], want_d[t]) is None, f"done differs at step {t}"
    assert (want_r != 0).any() or variant == "literal" or name == "c5"


# (workload, B, T) for multi-step launches: long enough that launches of 70 steps cross the
# engines' blocks of actions and results (16 steps on lane16, 64 on the wave and rows engines)
STEP_N_CASES = [("c1", 1, 150), ("c2", 203, 150), ("c3", 37, 80), ("c4", 333, 160),
                ("c5", 5, 75)]


@pytest.mark.parametrize("chunk", [7, 70])
@pytest.mark.parametrize("variant", ["literal", "dense"])
@pytest.mark.parametrize("engine", ["generic", "wave", "rows", "group", "auto"])
@pytest.mark.parametrize("case", STEP_N_CASES, ids=[f"{n}-B{b}-T{t}" for n, b, t in STEP_N_CASES])
def test_step_n_matches_oracle(case, engine, variant, chunk):
    require_gpu()
    name, B, T = case
    wl = inputs.WORKLOADS[name].with_(B=B, T=T, L=25)
    if engine == "group" and not group_ok(wl):
        pytest.skip("not eligible for the group engine")
    say(f"[parity step_n] {name} B={B} T={T} engine={engine} variant={variant} chunk={chunk}")
    maps, rules, actions = inputs.make_all(wl, 2, variant)
    want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8)
    _, final, r, d, _ = gpu_run(wl, maps, rules, actions, engine=engine, mode="step_n",
                                chunk=chunk)
    np.testing.assert_array_equal(r, want_r)
    np.testing.assert_array_equal(d, want_d)
    np.testing.assert_array_equal(final, want_m[-1])
    if T % 25 == 0:        # the last step is an episode-length reset step: check one before
        _, f2, _, _, _ = gpu_run(wl, maps, rules, actions[:T - 3], engine=engine, mode="step_n",
                                 chunk=chunk)
        np.testing.assert_array_equal(f2, want_m[T - 4])


# Shapes that stress the row-per-lane engine's edges: odd B (a half-empty lane word),
# maps narrower and shorter than 16, 1x1 up to 5x5 and 1x7 patterns, 2x2 maps.
EDGE = {
    "odd": inputs.Workload("odd", 31, B=77, H=5, W=11, C=5, R=6,
                           shapes=((1, 1), (2, 3), (4, 4), (3, 2)), p_dc=0.5, per_env=False,
                           T=30, L=7),
    "wide": inputs.Workload("wide", 32, B=40, H=16, W=16, C=9, R=10, shapes=((5, 5), (1, 7)),
                            p_dc=0.6, per_env=False, T=25, L=11),
    "tiny": inputs.Workload("tiny", 33, B=3, H=2, W=2, C=4, R=2, shapes=((1, 1), (2, 2)),
                            p_dc=0.4, per_env=False, T=20, L=0),
    "tall": inputs.Workload("tall", 34, B=9, H=16, W=3, C=6, R=4, shapes=((3, 1), (16, 1)),
                            p_dc=0.5, per_env=False, T=20, L=6),
}


@pytest.mark.parametrize("variant", inputs.VARIANTS)
@pytest.mark.parametrize("engine", ["generic", "lane16", "wave", "rows", "group"])
@pytest.mark.parametrize("name", sorted(EDGE))
def test_edge_shapes_match_oracle(name, engine, variant):
    require_gpu()
    wl = EDGE[name]
    if engine == "group" and not group_ok(wl):
        pytest.skip("not eligible for the group engine")
    say(f"[parity edge] {name} engine={engine} variant={variant}")
    maps, rules, actions = inputs.make_all(wl, 0, variant)
    want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8)
    seq, final, r, d, eng = gpu_run(wl, maps, rules, actions, engine=engine, mode="step")
    for t in range(wl.T):
        assert first_mismatch(seq[t], want_m[t]) is None, \
            f"maps differ at step {t}, index {first_mismatch(seq[t], want_m[t])}"
        np.testing.assert_array_equal(r[t], want_r[t], err_msg=f"rewards, step {t}")
        np.testing.assert_array_equal(d[t], want_d[t], err_msg=f"done, step {t}")
