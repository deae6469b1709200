"""av_step launches captured in a HIP graph (torch.cuda.graph on a side stream, the batch
switched to that stream with av_set_stream) and replayed: every replay, with eager work and
synchronisations in between, must give the maps, rewards and done flags of the same steps
taken eagerly, on every engine."""
import numpy as np
import pytest

import paper_2407_04221_amd as av
from gpu_util import require_gpu, say
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu

CASES = [("c4", 333, "lane16"), ("c2", 70, "rows"), ("c3", 9, "wave"), ("c5", 3, "rows"),
         ("c2", 21, "generic")]


@pytest.mark.parametrize("name,B,engine", CASES, ids=[f"{n}-{e}" for n, _, e in CASES])
def test_graph_replays_match_eager_steps(name, B, engine):
    require_gpu()
    import torch
    T = 12
    wl = inputs.WORKLOADS[name].with_(B=B, T=T, L=5)
    maps, rules, actions = inputs.make_all(wl, 1, "planted")
    acts = torch.from_numpy(actions).cuda()
    say(f"[graph] {name} B={B} engine={engine}")
    e = av.Batch.for_workload(wl, engine=engine)
    try:
        e.load_rules(*rules)
        e.reset(maps)
        want_r = torch.zeros((T, B), dtype=torch.float32, device="cuda")
        want_d = torch.zeros((T, B), dtype=torch.uint8, device="cuda")
        for t in range(T):
            av.av_step(e.h, acts[t], want_r[t], want_d[t])
        want_m = e.maps().cpu().numpy()
        want_r, want_d = want_r.cpu().numpy(), want_d.cpu().numpy()
    finally:
        e.close()
    assert (want_r != 0).any() and want_d.any()
    b = av.Batch.for_workload(wl, engine=engine)
    try:
        b.load_rules(*rules)
        b.reset(maps)
        rew = torch.zeros((T, B), dtype=torch.float32, device="cuda")
        don = torch.zeros((T, B), dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            av.av_set_stream(b.h, s)
            with torch.cuda.graph(g, stream=s):
                for t in range(T):
                    av.av_step(b.h, acts[t], rew[t], don[t])
        torch.cuda.current_stream().wait_stream(s)
        av.av_set_stream(b.h, torch.cuda.current_stream())
        assert b.info["engine"] == av.ENGINES[engine]
        for rep in range(3):
            b.reset(maps)                      # eager work between the replays
            rew.fill_(-7.0)
            don.fill_(9)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            np.testing.assert_array_equal(b.maps().cpu().numpy(), want_m, err_msg=f"maps, replay {rep}")
            np.testing.assert_array_equal(rew.cpu().numpy(), want_r, err_msg=f"rewards, replay {rep}")
            np.testing.assert_array_equal(don.cpu().numpy(), want_d, err_msg=f"done, replay {rep}")
    finally:
        b.close()
