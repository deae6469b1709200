"""Rule application control on the GPU (paper Sec. 2.1.1: capped, ordered or random site
selection and inhibition masks) vs the oracle: per-step maps, rewards and done flags for
every workload shape (cut down), both rule orders, both site orders; av_step_n launches
(the random channel follows the batch step number inside a launch); checkpoint and
resume mid-run; engine switching and argument errors."""
import numpy as np
import pytest

import oracle
from ctl_util import random_control
from gpu_util import first_mismatch, gpu_run, require_gpu, say
import paper_2407_04221_amd as av
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu

CASES = [("c1", 1, 40), ("c2", 37, 15), ("c3", 9, 12), ("c4", 77, 30), ("c5", 2, 6)]


def control_for(wl, B, seed, order, kmax=3):
    S = B if wl.per_env else 1
    limit, inhibit = random_control(np.random.default_rng(500 + seed), S, wl.R, kmax=kmax)
    return limit, inhibit, order, 0xC0FFEE + seed


@pytest.mark.parametrize("variant", ["planted", "dense"])
@pytest.mark.parametrize("order", [0, 1])
@pytest.mark.parametrize("mode", ["parallel", "sequential"])
@pytest.mark.parametrize("case", CASES, ids=[f"{n}-B{b}-T{t}" for n, b, t in CASES])
def test_control_step_matches_oracle(case, mode, order, variant):
    require_gpu()
    name, B, T = case
    wl = inputs.WORKLOADS[name].with_(B=B, T=T, L=9)
    say(f"[control] {name} mode={mode} order={order} variant={variant}")
    maps, rules, actions = inputs.make_all(wl, 4, variant)
    ctl = control_for(wl, B, 0, order)
    want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8,
                                        rule_mode=int(mode == "sequential"), control=ctl)
    seq, final, r, d, eng = gpu_run(wl, maps, rules, actions, engine="auto", mode="step",
                                    rule_mode=mode, control=ctl)
    lane16_ok = wl.H <= 16 and wl.W <= 16 and not wl.per_env
    assert av.ENGINE_NAMES[eng] == "lane16" if lane16_ok else av.ENGINE_NAMES[eng] in ("wave",
                                                                                        "generic")
    for t in range(T):
        assert first_mismatch(seq[t], want_m[t]) is None, \
            f"maps differ at step {t}, index {first_mismatch(seq[t], want_m[t])}"
        np.testing.assert_array_equal(r[t], want_r[t], err_msg=f"rewards, step {t}")
        np.testing.assert_array_equal(d[t], want_d[t], err_msg=f"done, step {t}")


WAVE_CASES = [("c2", 37, 12), ("c3", 9, 10), ("c5", 2, 6)]


@pytest.mark.parametrize("engine", ["wave", "generic"])
@pytest.mark.parametrize("order", [0, 1])
@pytest.mark.parametrize("mode", ["parallel", "sequential"])
@pytest.mark.parametrize("case", WAVE_CASES, ids=[c[0] for c in WAVE_CASES])
def test_control_explicit_engines(case, mode, order, engine):
    """The wave engine's control pass (and the generic engine's) on the per-environment and
    large-map workloads, dense rules, caps up to 4, in single steps and multi-step launches."""
    require_gpu()
    name, B, T = case
    wl = inputs.WORKLOADS[name].with_(B=B, T=T, L=8)
    say(f"[control {engine}] {name} mode={mode} order={order}")
    maps, rules, actions = inputs.make_all(wl, 8, "dense")
    ctl = control_for(wl, B, 4, order, kmax=4)
    try:
        want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8,
                                            rule_mode=int(mode == "sequential"), control=ctl)
        seq, final, r, d, eng = gpu_run(wl, maps, rules, actions, engine=engine, mode="step",
                                        rule_mode=mode, control=ctl)
    except av.AvError as e:
        # a wave batch whose control scratch does not fit its LDS refuses the control
        assert engine == "wave" and e.status == av.AV_EINVAL, e
        pytest.skip(str(e))
    assert av.ENGINE_NAMES[eng] == engine
    for t in range(T):
        assert first_mismatch(seq[t], want_m[t]) is None, f"maps differ at step {t}"
        np.testing.assert_array_equal(r[t], want_r[t], err_msg=f"rewards, step {t}")
        np.testing.assert_array_equal(d[t], want_d[t], err_msg=f"done, step {t}")
    _, final, r, d, _ = gpu_run(wl, maps, rules, actions, engine=engine, mode="step_n", chunk=5,
                                rule_mode=mode, control=ctl)
    np.testing.assert_array_equal(r, want_r)
    np.testing.assert_array_equal(d, want_d)
    np.testing.assert_array_equal(final, want_m[-1])


@pytest.mark.parametrize("order", [0, 1])
@pytest.mark.parametrize("case", CASES, ids=[f"{n}-B{b}-T{t}" for n, b, t in CASES])
def test_control_step_n_matches_oracle(case, order):
    require_gpu()
    name, B, T = case
    wl = inputs.WORKLOADS[name].with_(B=B, T=T, L=7)
    say(f"[control step_n] {name} order={order}")
    maps, rules, actions = inputs.make_all(wl, 5, "dense")
    ctl = control_for(wl, B, 1, order, kmax=6)
    want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8, control=ctl)
    _, final, r, d, _ = gpu_run(wl, maps, rules, actions, engine="generic", mode="step_n",
                                chunk=4, control=ctl)
    np.testing.assert_array_equal(r, want_r)
    np.testing.assert_array_equal(d, want_d)
    np.testing.assert_array_equal(final, want_m[-1])


LANE16_CASES = [("c1", 1, 40), ("c4", 77, 30),
                ("sq16", 45, 20), ("odd", 29, 25)]
LANE16_EXTRA = {
    "sq16": inputs.Workload("sq16", 63, B=45, H=16, W=16, C=7, R=9,
                            shapes=((3, 3), (1, 2), (4, 1)), p_dc=0.5, per_env=False, T=20, L=7),
    "odd": inputs.Workload("odd", 61, B=29, H=5, W=11, C=5, R=6,
                           shapes=((1, 1), (2, 3), (3, 2)), p_dc=0.5, per_env=False, T=25, L=6),
}


@pytest.mark.parametrize("order", [0, 1])
@pytest.mark.parametrize("variant", ["planted", "dense"])
@pytest.mark.parametrize("mode", ["parallel", "sequential"])
@pytest.mark.parametrize("case", LANE16_CASES, ids=[c[0] for c in LANE16_CASES])
def test_lane16_control_matches_oracle(case, mode, variant, order):
    """Caps (row-major and random order) and inhibition compiled into the lane16 program,
    stepped one launch per step and in multi-step launches (the random channel follows the
    batch step number inside a launch)."""
    require_gpu()
    name, B, T = case
    wl = LANE16_EXTRA[name] if name in LANE16_EXTRA else inputs.WORKLOADS[name].with_(B=B, T=T,
                                                                                      L=9)
    say(f"[lane16 control] {name} mode={mode} variant={variant} order={order}")
    maps, rules, actions = inputs.make_all(wl, 6, variant)
    for kmax, seed in ((1, 0), (4, 1)):
        ctl = control_for(wl, wl.B, seed, order, kmax=kmax)
        want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8,
                                            rule_mode=int(mode == "sequential"), control=ctl)
        seq, final, r, d, eng = gpu_run(wl, maps, rules, actions, engine="lane16", mode="step",
                                        rule_mode=mode, control=ctl)
        assert av.ENGINE_NAMES[eng] == "lane16"
        for t in range(wl.T):
            assert first_mismatch(seq[t], want_m[t]) is None, f"kmax {kmax}: maps differ, step {t}"
            np.testing.assert_array_equal(r[t], want_r[t], err_msg=f"kmax {kmax}: rewards {t}")
            np.testing.assert_array_equal(d[t], want_d[t], err_msg=f"kmax {kmax}: done {t}")
        _, final, r, d, _ = gpu_run(wl, maps, rules, actions, engine="lane16", mode="step_n",
                                    chunk=6, rule_mode=mode, control=ctl)
        np.testing.assert_array_equal(r, want_r)
        np.testing.assert_array_equal(d, want_d)
        np.testing.assert_array_equal(final, want_m[-1])


def test_control_full_size_c4_prefix():
    """c4 at its full batch (16384 environments) with random-order limits and inhibition:
    the first 256 environments checked against the oracle every step (the random channel
    depends on the environment index, so the oracle gets the same leading indices)."""
    require_gpu()
    import torch
    wl = inputs.WORKLOADS["c4"].with_(T=20)
    say(f"[control full] c4 B={wl.B} T={wl.T}")
    maps, rules, actions = inputs.make_all(wl, 0, "dense")
    ctl = control_for(wl, wl.B, 2, 1, kmax=4)
    n = 256
    want_m, want_r, want_d = oracle.run(wl, maps[:n], rules, actions[:, :n], nthreads=8,
                                        B=n, control=ctl)
    b = av.Batch.for_workload(wl)
    try:
        b.load_rules(*rules)
        b.set_rule_control(*ctl)
        b.reset(maps)
        acts = torch.from_numpy(actions).cuda()
        for t in range(wl.T):
            r, d = b.step(acts[t])
            got = b.maps()[:n].cpu().numpy()
            assert first_mismatch(got, want_m[t]) is None, f"step {t}"
            np.testing.assert_array_equal(r[:n].cpu().numpy(), want_r[t])
            np.testing.assert_array_equal(d[:n].cpu().numpy(), want_d[t])
    finally:
        b.close()


@pytest.mark.parametrize("name", ["c2", "c4"])
def test_control_checkpoint_resume(name):
    """The blob carries the batch step number: resuming from it repeats the random picks
    (generic engine for c2's per-environment rules, lane16 for c4)."""
    require_gpu()
    import torch
    wl = inputs.WORKLOADS[name].with_(B=40, T=12, L=50)
    maps, rules, actions = inputs.make_all(wl, 1, "dense")
    ctl = control_for(wl, wl.B, 3, 1)
    acts = torch.from_numpy(actions).cuda()

    def make():
        b = av.Batch.for_workload(wl)
        b.load_rules(*rules)
        b.set_rule_control(*ctl)
        b.reset(maps)
        return b

    a = make()
    for t in range(5):
        a.step(acts[t])
    blob = a.get_state()
    tail = []
    for t in range(5, wl.T):
        r, d = a.step(acts[t])
        tail.append((a.maps().cpu().numpy(), r.cpu().numpy().copy()))
    a.close()
    c = make()
    c.set_state(blob)
    for k, t in enumerate(range(5, wl.T)):
        r, d = c.step(acts[t])
        np.testing.assert_array_equal(c.maps().cpu().numpy(), tail[k][0])
        np.testing.assert_array_equal(r.cpu().numpy(), tail[k][1])
    c.close()


def test_control_engine_switch_and_errors():
    require_gpu()
    wl = inputs.WORKLOADS["c4"].with_(B=8, T=1)
    maps, rules, actions = inputs.make_all(wl, 0, "planted")
    R = wl.R
    b = av.Batch.for_workload(wl)
    try:
        with pytest.raises(av.AvError) as e:
            b.set_rule_control(None, None, "rowmajor", 0)
        assert e.value.status == av.AV_ESTATE
        b.load_rules(*rules)
        assert b.info["engine"] == av.AV_ENGINE_LANE16
        lim = np.zeros((1, R), np.int32)
        b.set_rule_control(lim, None, "random", 1)          # nothing active: engine kept
        assert b.info["engine"] == av.AV_ENGINE_LANE16
        lim[0, 2] = 1
        b.set_rule_control(lim, None, "rowmajor", 0)           # compiled into lane16
        assert b.info["engine"] == av.AV_ENGINE_LANE16
        b.set_rule_control(lim, None, "random", 0)             # so is the random order
        assert b.info["engine"] == av.AV_ENGINE_LANE16
        b.set_rule_control(None, None)
        assert b.info["engine"] == av.AV_ENGINE_LANE16
    finally:
        b.close()
    b = av.Batch.for_workload(wl, engine="generic")
    try:
        b.load_rules(*rules)
        b.set_rule_control(np.ones((1, R), np.int32), None, "random", 0)
        assert b.info["engine"] == av.AV_ENGINE_GENERIC
    finally:
        b.close()
    b = av.Batch.for_workload(wl)
    try:
        b.load_rules(*rules)
        b.set_rule_control(lim, None)
        b.load_rules(*rules)                                 # clears the control
        assert b.info["engine"] == av.AV_ENGINE_LANE16
        bad = np.zeros((1, R), np.int32)
        bad[0, 0] = -2
        inh = np.zeros((1, R, R), np.uint8)
        inh[0, 3, 3] = 1
        inh2 = np.zeros((1, R, R), np.uint8)
        inh2[0, 5, 1] = 1
        for args in ((bad, None, 0, 0), (None, inh, 0, 0), (None, inh2, 0, 0),
                     (None, None, 2, 0)):
            with pytest.raises(av.AvError) as e:
                av.av_set_rule_control(b.h, *args)
            assert e.value.status == av.AV_EINVAL
    finally:
        b.close()
    b = av.Batch.for_workload(wl, engine="lane16")
    try:
        b.load_rules(*rules)
        lim = np.ones((1, R), np.int32)
        b.set_rule_control(lim, None)                          # both orders run on lane16
        b.set_rule_control(lim, None, "random", 0)
        assert b.info["engine"] == av.AV_ENGINE_LANE16
    finally:
        b.close()
    b = av.Batch.for_workload(wl, engine="wave")
    try:
        b.load_rules(*rules)
        b.set_rule_control(np.ones((1, R), np.int32), None)    # the wave engine runs it
        assert b.info["engine"] == av.AV_ENGINE_WAVE
    finally:
        b.close()


def test_control_on_rows_batches():
    """An AUTO batch on the rows engine runs rule application control on the wave engine and
    returns to rows when the control is cleared; an explicit rows batch refuses it; both
    against the oracle."""
    require_gpu()
    wl = inputs.WORKLOADS["c5"].with_(B=3, T=6, L=5)
    maps, rules, actions = inputs.make_all(wl, 8, "dense")
    ctl = control_for(wl, 3, 4, 0, kmax=3)
    R = wl.R
    b = av.Batch.for_workload(wl)
    try:
        b.load_rules(*rules)
        assert b.info["engine"] == av.AV_ENGINE_ROWS
        b.set_rule_control(*ctl)
        assert b.info["engine"] == av.AV_ENGINE_WAVE
        b.set_rule_control(None, None)
        assert b.info["engine"] == av.AV_ENGINE_ROWS
    finally:
        b.close()
    b = av.Batch.for_workload(wl, engine="rows")
    try:
        b.load_rules(*rules)
        with pytest.raises(av.AvError) as e:
            b.set_rule_control(np.ones((1, R), np.int32), None)
        assert e.value.status == av.AV_EINVAL
        b.set_rule_control(np.zeros((1, R), np.int32), None)     # no control: accepted
        assert b.info["engine"] == av.AV_ENGINE_ROWS
    finally:
        b.close()
    want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8, control=ctl)
    seq, final, r, d, eng = gpu_run(wl, maps, rules, actions, engine="auto", mode="step",
                                    control=ctl)
    assert av.ENGINE_NAMES[eng] == "wave"
    for t in range(wl.T):
        assert first_mismatch(seq[t], want_m[t]) is None, f"maps differ at step {t}"
        np.testing.assert_array_equal(r[t], want_r[t], err_msg=f"rewards, step {t}")
        np.testing.assert_array_equal(d[t], want_d[t], err_msg=f"done, step {t}")
