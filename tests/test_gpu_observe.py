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
