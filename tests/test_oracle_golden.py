"""Oracle pinned to hand-worked cases (tests/golden/*.av): each fixture's expected maps,
rewards and done flags were derived by hand from the paper's text (citations inside the
fixtures).  The convolution form of the step (Sec. 2.1) is checked on the same cases."""
import numpy as np
import pytest

import e3_conv
import fixtures
import oracle

FIXTURES = fixtures.all_fixtures()


def _ids(paths):
    return [p.rsplit("/", 1)[-1][:-3] for p in paths]


def run_oracle(fx):
    shape, ip, op, rw, mh, mw = fx.abi_rules()
    o = oracle.Oracle(1, fx.H, fx.W, fx.C, max(len(fx.rules), 1), mh, mw, False, fx.L,
                      rule_mode=fx.mode)
    o.load_rules(shape, ip, op, rw)
    if fx.has_control:
        o.set_rule_control(*fx.abi_control())
    o.reset(fx.init[None])
    got = []
    for st in fx.steps:
        r, d = o.step(np.array([st.action], np.uint8))
        got.append((o.maps()[0], float(r[0]), int(d[0])))
    o.close()
    return got


@pytest.mark.parametrize("path", FIXTURES, ids=_ids(FIXTURES))
def test_oracle_matches_worked_case(oracle_lib, path):
    fx = fixtures.parse(path)
    assert fx.steps, "fixture without steps"
    for k, (st, (m, r, d)) in enumerate(zip(fx.steps, run_oracle(fx))):
        np.testing.assert_array_equal(m, st.after, err_msg=f"{fx.name} step {k} map")
        assert r == st.reward, f"{fx.name} step {k} reward {r} != {st.reward}"
        assert d == st.done, f"{fx.name} step {k} done {d} != {st.done}"


@pytest.mark.parametrize("path", FIXTURES, ids=_ids(FIXTURES))
def test_conv_form_matches_worked_case(path):
    fx = fixtures.parse(path)
    shape, ip, op, rw, _, _ = fx.abi_rules()
    acts = np.array([[st.action] for st in fx.steps], np.uint8)
    maps, rewards, done = e3_conv.run(fx.init[None], (shape, ip, op, rw), acts, L=fx.L,
                                      sequential=bool(fx.mode),
                                      control=fx.abi_control() if fx.has_control else None)
    for k, st in enumerate(fx.steps):
        np.testing.assert_array_equal(maps[k, 0], st.after, err_msg=f"{fx.name} step {k}")
        assert rewards[k, 0] == st.reward
        assert done[k, 0] == st.done


def test_fixture_set_is_complete():
    names = set(_ids(FIXTURES))
    # a single rule firing, a don't-care cell, overlapping matches, a move into a wall
    for need in ("w01_single_rule", "w02_dont_care", "w03_overlap", "w04_move_into_wall",
                 "w06_food", "w07_kill", "w08_edge", "w10_vote_count", "ws01_food_sequential",
                 "ws02_chain_sequential", "wc01_once_rowmajor", "wc03_inhibit_overlap",
                 "wc04_inhibit_2d"):
        assert need in names
