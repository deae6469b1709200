"""The group engine on a batch larger than the GPU's SIMDs: after launches of 64 steps or more
it reorders which workgroup steps which environment by the cycles each environment took (the
slowest one per SIMD, the lightest beside them), so the order changes from launch to launch.
Rewards, done flags and maps must not change: they are compared with the oracle after every
launch.  The launches are separated by a synchronization, so each one after the first runs in
the order computed from the launch before; 1500 environments fill one wave per SIMD of a
1024-SIMD GPU and part of a second."""
import numpy as np
import pytest

import oracle
from gpu_util import first_mismatch, group_ok, require_gpu, say
import paper_2407_04221_amd as av
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("variant", ["literal", "planted", "dense"])
def test_results_do_not_depend_on_the_workgroup_order(variant):
    import torch
    require_gpu()
    wl = inputs.Workload("order", 61, B=1500, H=16, W=16, C=6, R=8, shapes=((3, 3), (1, 2)),
                         p_dc=0.3, per_env=True, T=300, L=45)
    assert group_ok(wl)
    say(f"[group order] B={wl.B} variant={variant}")
    maps, rules, actions = inputs.make_all(wl, 5, variant)
    o = oracle.Oracle.for_workload(wl)
    o.load_rules(*rules)
    o.reset(maps)
    b = av.Batch.for_workload(wl, engine="group")
    try:
        b.load_rules(*rules)
        b.reset(maps)
        assert b.info["engine"] == av.AV_ENGINE_GROUP
        acts = torch.from_numpy(np.ascontiguousarray(actions)).cuda()
        rew = torch.empty((wl.T, wl.B), dtype=torch.float32, device="cuda")
        don = torch.empty((wl.T, wl.B), dtype=torch.uint8, device="cuda")
        for t0 in range(0, wl.T, 100):
            b.step_n(acts[t0:t0 + 100], rew[t0:t0 + 100], don[t0:t0 + 100])
            torch.cuda.synchronize()
            for t in range(t0, t0 + 100):
                want_r, want_d = o.step(actions[t], 8)
                np.testing.assert_array_equal(rew[t].cpu().numpy(), want_r, err_msg=f"rewards, step {t}")
                np.testing.assert_array_equal(don[t].cpu().numpy(), want_d, err_msg=f"done, step {t}")
            got, want = b.maps().cpu().numpy(), o.maps()
            assert first_mismatch(got, want) is None, \
                f"maps differ after step {t0 + 99}, index {first_mismatch(got, want)}"
    finally:
        b.close()
        o.close()


def test_captured_launch_replays_under_a_changing_order():
    """A captured av_step_n of 64 steps on such a batch: capture leaves the order alone, while
    the eager launches between the replays reorder the workgroups, so replays run under orders
    the capture never saw; every launch is compared with the oracle."""
    import torch
    require_gpu()
    wl = inputs.Workload("order_graph", 62, B=1300, H=16, W=16, C=6, R=8,
                         shapes=((3, 3), (1, 2)), p_dc=0.3, per_env=True, T=64, L=40)
    maps, rules, actions = inputs.make_all(wl, 6, "planted")
    say(f"[group order graph] B={wl.B}")
    o = oracle.Oracle.for_workload(wl)
    o.load_rules(*rules)
    o.reset(maps)
    b = av.Batch.for_workload(wl, engine="group")
    try:
        b.load_rules(*rules)
        b.reset(maps)
        acts = torch.from_numpy(np.ascontiguousarray(actions)).cuda()   # one block of 64 steps
        rew = torch.empty((64, wl.B), dtype=torch.float32, device="cuda")
        don = torch.empty((64, wl.B), dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        try:
            with torch.cuda.stream(s):
                av.av_set_stream(b.h, s)
                with torch.cuda.graph(g, stream=s):
                    av.av_step_n(b.h, 64, acts, rew, don)
        finally:
            torch.cuda.current_stream().wait_stream(s)
            av.av_set_stream(b.h, torch.cuda.current_stream())
        for n, how in enumerate(("eager", "eager", "replay", "eager", "replay", "replay")):
            if how == "eager":
                b.step_n(acts, rew, don)
            else:
                g.replay()
            torch.cuda.synchronize()
            for t in range(64):
                want_r, want_d = o.step(actions[t], 8)
                np.testing.assert_array_equal(rew[t].cpu().numpy(), want_r,
                                              err_msg=f"launch {n} ({how}): rewards, step {t}")
                np.testing.assert_array_equal(don[t].cpu().numpy(), want_d,
                                              err_msg=f"launch {n} ({how}): done, step {t}")
            got, want = b.maps().cpu().numpy(), o.maps()
            assert first_mismatch(got, want) is None, \
                f"launch {n} ({how}): maps differ at {first_mismatch(got, want)}"
    finally:
        b.close()
        o.close()
