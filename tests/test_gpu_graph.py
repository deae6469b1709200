"""av_step launches captured in a HIP graph (torch.cuda.graph on a side stream, the batch
switched to that stream with av_set_stream) and replayed, checked against the oracle.

The graph holds one av_step.  It is replayed once per step with no reset in between, and the
maps (read eagerly with av_get_maps), rewards and done flags after every replay must equal
the oracle's trajectory; then the batch is reset eagerly and the same graph replayed again,
which must follow the oracle from the reset.  With rule application control in random site
order (paper Sec. 2.1.1), the random index channel is keyed on the batch step number: every
replay must advance it on the device, or replays would repeat the captured step's keys."""
import numpy as np
import pytest

import oracle
import paper_2407_04221_amd as av
from ctl_util import random_control
from gpu_util import first_mismatch, require_gpu, say
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu

# (workload, B, engine, control): control None, or the site order of a random cap/inhibition
CASES = [("c4", 333, "lane16", None), ("c2", 70, "rows", None), ("c3", 9, "wave", None),
         ("c5", 3, "rows", None), ("c2", 21, "generic", None), ("c2", 70, "group", None),
         ("c3", 9, "group", None),
         ("c4", 333, "lane16", "random"), ("c4", 77, "lane16", "rowmajor"),
         ("c2", 37, "wave", "random"), ("c3", 9, "generic", "random"),
         ("c5", 2, "generic", "random")]


def _ids():
    return [f"{n}-B{b}-{e}" + (f"-{c}" if c else "") for n, b, e, c in CASES]


def _capture_one_step(torch, b, act, rew, don):
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    try:
        with torch.cuda.stream(s):
            av.av_set_stream(b.h, s)
            with torch.cuda.graph(g, stream=s):
                av.av_step(b.h, act, rew, don)
    finally:
        torch.cuda.current_stream().wait_stream(s)
        av.av_set_stream(b.h, torch.cuda.current_stream())
    return g


@pytest.mark.parametrize("name,B,engine,order", CASES, ids=_ids())
def test_graph_replays_match_oracle(name, B, engine, order):
    require_gpu()
    import torch
    T1, T2 = 14, 9
    wl = inputs.WORKLOADS[name].with_(B=B, T=T1, L=5)
    if name == "c5" and order:
        # c5's own 5 x 5 rules over 13 channels rarely match; small patterns make the caps bind
        wl = wl.with_(shapes=((1, 1), (1, 2), (2, 2)))
    variant = "dense" if order else "planted"
    maps, rules, actions = inputs.make_all(wl, 1, variant)
    # one action row for every step: the graph reads the same action buffer each replay
    acts_np = np.ascontiguousarray(np.broadcast_to(actions[0], (T1, B)))
    ctl = None
    if order:
        S = B if wl.per_env else 1
        limit, inhibit = random_control(np.random.default_rng(77), S, wl.R, kmax=2)
        limit[limit == 0] = 1
        ctl = (limit, inhibit, av.SITE_ORDERS[order], 0xBEEF)
    say(f"[graph] {name} B={B} engine={engine} control={order}")
    want_m, want_r, want_d = oracle.run(wl, maps, rules, acts_np, nthreads=8, control=ctl)
    want2_m, want2_r, want2_d = oracle.run(wl, maps, rules, acts_np[:T2], nthreads=8,
                                           control=ctl)
    assert (want_r != 0).any() and want_d.any()
    b = av.Batch.for_workload(wl, engine=engine)
    try:
        b.load_rules(*rules)
        if ctl is not None:
            b.set_rule_control(*ctl)
        b.reset(maps)
        act = torch.from_numpy(acts_np[0].copy()).cuda()
        rew = torch.zeros(B, dtype=torch.float32, device="cuda")
        don = torch.zeros(B, dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        g = _capture_one_step(torch, b, act, rew, don)
        assert b.info["engine"] == av.ENGINES[engine]
        for phase, (T, wm, wr, wd) in enumerate(((T1, want_m, want_r, want_d),
                                                 (T2, want2_m, want2_r, want2_d))):
            if phase == 1:
                b.reset(maps)                  # eager work between the replays
            for t in range(T):
                rew.fill_(-7.0)
                don.fill_(9)
                torch.cuda.synchronize()
                g.replay()
                torch.cuda.synchronize()
                got = b.maps().cpu().numpy()
                assert first_mismatch(got, wm[t]) is None, \
                    f"phase {phase}: maps differ after replay {t} at {first_mismatch(got, wm[t])}"
                np.testing.assert_array_equal(rew.cpu().numpy(), wr[t],
                                              err_msg=f"phase {phase}: rewards, replay {t}")
                np.testing.assert_array_equal(don.cpu().numpy(), wd[t],
                                              err_msg=f"phase {phase}: done, replay {t}")
    finally:
        b.close()


def test_graph_of_step_n_launches_matches_oracle():
    """A graph of three av_step_n launches (5, 1 and 17 steps) on lane16 with a random cap,
    replayed twice without a reset: the launches' batch step numbers advance on the device."""
    require_gpu()
    import torch
    wl = inputs.WORKLOADS["c4"].with_(B=129, T=46, L=7)
    maps, rules, actions = inputs.make_all(wl, 3, "dense")
    limit, inhibit = random_control(np.random.default_rng(5), 1, wl.R, kmax=3)
    limit[limit == 0] = 2
    ctl = (limit, inhibit, av.AV_SITES_RANDOM, 99)
    half = np.ascontiguousarray(actions[:23])
    acts2 = np.concatenate([half, half])       # the graph replays the same 23 action rows
    want_m, want_r, want_d = oracle.run(wl, maps, rules, acts2, nthreads=8, control=ctl)
    b = av.Batch.for_workload(wl, engine="lane16")
    try:
        b.load_rules(*rules)
        b.set_rule_control(*ctl)
        b.reset(maps)
        acts = torch.from_numpy(half).cuda()
        rew = torch.zeros((23, wl.B), dtype=torch.float32, device="cuda")
        don = torch.zeros((23, wl.B), dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        try:
            with torch.cuda.stream(s):
                av.av_set_stream(b.h, s)
                with torch.cuda.graph(g, stream=s):
                    for lo, hi in ((0, 5), (5, 6), (6, 23)):
                        av.av_step_n(b.h, hi - lo, acts[lo:hi], rew[lo:hi], don[lo:hi])
        finally:
            torch.cuda.current_stream().wait_stream(s)
            av.av_set_stream(b.h, torch.cuda.current_stream())
        for rep in range(2):
            g.replay()
            torch.cuda.synchronize()
            sl = slice(23 * rep, 23 * rep + 23)
            np.testing.assert_array_equal(rew.cpu().numpy(), want_r[sl], err_msg=f"replay {rep}")
            np.testing.assert_array_equal(don.cpu().numpy(), want_d[sl], err_msg=f"replay {rep}")
            np.testing.assert_array_equal(b.maps().cpu().numpy(), want_m[23 * rep + 22],
                                          err_msg=f"maps, replay {rep}")
    finally:
        b.close()
