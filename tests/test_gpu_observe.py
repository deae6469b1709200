"""Observation on the GPU vs the oracle: after some steps of each workload (cut down), the
player-centred windows for several sizes, and the binary rule features."""
import numpy as np
import pytest

import oracle
import paper_2407_04221_amd as av
from gpu_util import require_gpu, say
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu

CASES = [("c1", 1, 9), ("c2", 130, 7), ("c3", 17, 5), ("c4", 301, 11), ("c5", 3, 4)]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_observe_matches_oracle(case):
    require_gpu()
    import torch
    name, B, T = case
    wl = inputs.WORKLOADS[name].with_(B=B, T=T, L=5)
    maps, rules, actions = inputs.make_all(wl, 1, "planted")
    o = oracle.Oracle.for_workload(wl)
    o.load_rules(*rules)
    o.reset(maps)
    b = av.Batch.for_workload(wl)
    b.load_rules(*rules)
    b.reset(maps)
    acts = torch.from_numpy(actions).cuda()
    for t in range(T):
        o.step(actions[t])
    b.step_n(acts)
    wins = (1, 2, 5, 10, 20, 31, 2 * wl.H + 3) + ((100,) if wl.H <= 16 else ())
    for w in wins:
        say(f"[observe] {name} w={w}")
        np.testing.assert_array_equal(b.observe(w).cpu().numpy(), o.observe(w), err_msg=f"w={w}")
    o.close()
    b.close()


@pytest.mark.parametrize("per_env", [False, True])
def test_rule_features_match_oracle(per_env):
    require_gpu()
    import torch
    wl = inputs.Workload("feat", 71, B=9, H=8, W=9, C=5, R=4, shapes=((3, 3), (1, 2)), p_dc=0.4,
                         per_env=per_env, T=1)
    maps, (shape, ip, op, rw), _ = inputs.make_all(wl, 0)
    o = oracle.Oracle.for_workload(wl)
    o.load_rules(shape, ip, op, rw)
    want = o.rule_features(wl.S, wl.R)
    o.close()
    b = av.Batch.for_workload(wl)
    dst = torch.empty(want.shape, dtype=torch.uint8, device="cuda")
    with pytest.raises(av.AvError) as e:
        av.av_rule_features(b.h, dst)
    assert e.value.status == av.AV_ESTATE
    b.load_rules(shape, ip, op, rw)
    av.av_rule_features(b.h, dst)
    np.testing.assert_array_equal(dst.cpu().numpy(), want)
    b.close()


def test_observe_rejects_bad_window():
    require_gpu()
    import torch
    wl = inputs.WORKLOADS["c1"]
    maps, rules, _ = inputs.make_all(wl, 0)
    b = av.Batch.for_workload(wl)
    b.load_rules(*rules)
    dst = torch.empty((1, wl.C, 5, 5), dtype=torch.uint8, device="cuda")
    with pytest.raises(av.AvError) as e:
        av.av_observe(b.h, 5, dst)
    assert e.value.status == av.AV_ESTATE        # no maps yet
    b.reset(maps)
    lib = av.load_library()
    import ctypes
    assert lib.av_observe(b.h, 0, ctypes.c_void_p(dst.data_ptr())) == av.AV_EINVAL
    assert lib.av_observe(b.h, 256, ctypes.c_void_p(dst.data_ptr())) == av.AV_EINVAL
    b.close()


STEP_OBS = [("c1", 1, 6), ("c2", 70, 5), ("c4", 301, 7), ("c4", 13, 4), ("c5", 2, 4)]


@pytest.mark.parametrize("engine", ["auto", "lane16", "generic", "wave", "rows"])
@pytest.mark.parametrize("case", STEP_OBS, ids=[f"{c[0]}-B{c[1]}" for c in STEP_OBS])
def test_step_observe_matches_oracle(case, engine):
    """av_step_observe (the observation written by the lane16 step kernel itself for w <= 64,
    else the observation kernel after the step) against the oracle stepping then observing,
    after every call, with one and several steps per call."""
    require_gpu()
    import torch
    name, B, T = case
    wl = inputs.WORKLOADS[name].with_(B=B, T=T, L=4)
    lane16_ok = wl.H <= 16 and wl.W <= 16 and not wl.per_env
    if engine == "lane16" and not lane16_ok:
        pytest.skip("lane16 takes maps of at most 16 x 16 with one shared rule set")
    maps, rules, actions = inputs.make_all(wl, 2, "planted")
    wins = (1, 2, 5, 10, 20, 31, 64) + ((100,) if wl.H <= 16 else ())
    for w in wins:
        say(f"[step_observe] {name} B={B} engine={engine} w={w}")
        o = oracle.Oracle.for_workload(wl)
        o.load_rules(*rules)
        o.reset(maps)
        b = av.Batch.for_workload(wl, engine=engine)
        b.load_rules(*rules)
        b.reset(maps)
        acts = torch.from_numpy(actions).cuda()
        t = 0
        for k in (1, 2, T - 3):
            want_r = np.zeros((k, wl.B), np.float32)
            want_d = np.zeros((k, wl.B), np.uint8)
            for j in range(k):
                want_r[j], want_d[j] = o.step(actions[t + j])
            r, d, obs = b.step_observe(acts[t:t + k], w)
            t += k
            np.testing.assert_array_equal(r.cpu().numpy(), want_r, err_msg=f"w={w} rewards")
            np.testing.assert_array_equal(d.cpu().numpy(), want_d, err_msg=f"w={w} done")
            np.testing.assert_array_equal(b.maps().cpu().numpy(), o.maps(), err_msg=f"w={w} maps")
            np.testing.assert_array_equal(obs.cpu().numpy(), o.observe(w), err_msg=f"w={w} obs")
        o.close()
        b.close()


@pytest.mark.parametrize("w", [5, 12])
def test_step_observe_with_random_control(w):
    """The fused observation next to the random-order control's LDS keys (w = 5 fits both in
    LDS; w = 12 falls back to the observation kernel)."""
    require_gpu()
    import torch
    from ctl_util import random_control
    wl = inputs.WORKLOADS["c4"].with_(B=77, T=6, L=4)
    maps, rules, actions = inputs.make_all(wl, 3, "dense")
    limit, inhibit = random_control(np.random.default_rng(9), 1, wl.R, kmax=3)
    ctl = (limit, inhibit, 1, 77)
    o = oracle.Oracle.for_workload(wl)
    o.load_rules(*rules)
    o.set_rule_control(*ctl)
    o.reset(maps)
    b = av.Batch.for_workload(wl)
    b.load_rules(*rules)
    b.set_rule_control(*ctl)
    b.reset(maps)
    assert b.info["engine"] == av.AV_ENGINE_LANE16
    acts = torch.from_numpy(actions).cuda()
    for t in range(wl.T):
        want_r, want_d = o.step(actions[t])
        r, d, obs = b.step_observe(acts[t:t + 1], w)
        np.testing.assert_array_equal(r.cpu().numpy()[0], want_r)
        np.testing.assert_array_equal(d.cpu().numpy()[0], want_d)
        np.testing.assert_array_equal(obs.cpu().numpy(), o.observe(w), err_msg=f"step {t}")
    o.close()
    b.close()


def test_observe_without_player_several_players_and_unaligned_output():
    """Maps with no player (all-zero windows), several players (the first in row-major order
    centres the window), and an output that starts 3 bytes past a 16-byte boundary."""
    require_gpu()
    import torch
    wl = inputs.Workload("obsedge", 72, B=11, H=13, W=10, C=5, R=1, shapes=((1, 1),), p_dc=0.5,
                         per_env=False, T=1)
    maps, rules, _ = inputs.make_all(wl, 0)
    maps[::3, 2] = 0                              # no player
    maps[1::3, 2, 4, 7] = 1                       # a second player
    maps[1::3, 2, 9, 0] = 1                       # and a third
    o = oracle.Oracle.for_workload(wl)
    o.load_rules(*rules)
    o.reset(maps)
    b = av.Batch.for_workload(wl)
    b.load_rules(*rules)
    b.reset(maps)
    for w in (1, 3, 7, 16, 29):
        n = wl.B * wl.C * w * w
        buf = torch.full((n + 40,), 7, dtype=torch.uint8, device="cuda")
        dst = buf[3:3 + n].view(wl.B, wl.C, w, w)
        av.av_observe(b.h, w, dst)
        want = o.observe(w)
        assert not want[::3].any()
        np.testing.assert_array_equal(dst.cpu().numpy(), want, err_msg=f"w={w}")
        rest = buf.cpu().numpy()
        assert (rest[:3] == 7).all() and (rest[3 + n:] == 7).all(), "wrote outside the output"
    o.close()
    b.close()
