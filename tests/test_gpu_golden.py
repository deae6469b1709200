"""Every hand-worked fixture (tests/golden/*.av, derived from the paper's text) run through
each eligible GPU engine: the GPU is checked against the hand-worked values directly, not
only against the oracle."""
import numpy as np
import pytest

import fixtures
from gpu_util import gpu_run, require_gpu, say
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu

FIXTURES = fixtures.all_fixtures()


def _cases():
    out = []
    for path in FIXTURES:
        fx = fixtures.parse(path)
        name = path.rsplit("/", 1)[-1][:-3]
        if fx.has_control:      # rule application control: generic and lane16
            engines = ["generic", "auto"]
            if fx.H <= 16 and fx.W <= 16:
                engines.append("lane16")
        else:
            engines = ["generic", "wave", "rows"]
            if fx.H <= 16 and fx.W <= 16:
                engines.append("lane16")
        out += [(name, path, e) for e in engines]
    return out


@pytest.mark.parametrize("name,path,engine", _cases(), ids=[f"{n}-{e}" for n, _, e in _cases()])
def test_gpu_matches_worked_case(name, path, engine):
    require_gpu()
    fx = fixtures.parse(path)
    shape, ip, op, rw, mh, mw = fx.abi_rules()
    R = len(fx.rules)
    wl = inputs.Workload(name, 0, B=1, H=fx.H, W=fx.W, C=fx.C, R=R, shapes=((mh, mw),),
                         p_dc=0.0, per_env=False, T=len(fx.steps), L=fx.L)
    acts = np.array([[st.action] for st in fx.steps], np.uint8)
    say(f"[golden] {name} engine={engine}")
    seq, final, r, d, _ = gpu_run(wl, fx.init[None], (shape, ip, op, rw), acts, engine=engine,
                                  mode="step", rule_mode="sequential" if fx.mode else "parallel",
                                  control=fx.abi_control() if fx.has_control else None)
    for k, st in enumerate(fx.steps):
        np.testing.assert_array_equal(seq[k][0], st.after, err_msg=f"{name} step {k}")
        assert r[k, 0] == st.reward, f"{name} step {k} reward"
        assert d[k, 0] == st.done, f"{name} step {k} done"
