"""Oracle rule application control (paper Sec. 2.1.1: a rule can be made to apply only once
or a fixed number of times, in an ordered or a random order, by taking the maximum over an
extra channel of index values; masks can make some rules inhibit others), pinned by:

  * the Philox4x64-10 block function against numpy's independent implementation;
  * the hand-worked fixtures tests/golden/wc*.av (run by test_oracle_golden);
  * an independent formulation (tests/e3_conv.py): matches from the convolution form,
    inhibition as a convolution of the inhibitor's applied anchors with a box of ones,
    selection with numpy's Philox and argsort;
  * closed forms: a rule that matches everywhere, limited to K, applies at exactly K
    anchors (the first K in row-major order for the ordered channel);
  * planted mistakes in the oracle that these pins must catch.
"""
import os

import numpy as np
import pytest

import e3_conv
import fixtures
from ctl_util import random_control
import oracle
from paper_2407_04221_amd import inputs

P = 2


@pytest.mark.parametrize("ctr,key", [
    ((0, 0, 0, 0), (0, 0)),
    ((1, 0, 0, 0), (0, 0)),
    ((7, 123456789, 42, 0), (0xDEADBEEF, 0)),
    ((2**64 - 1, 2**64 - 1, 2**64 - 1, 2**64 - 1), (2**64 - 1, 2**64 - 1)),
    ((511, 10**12, 16383, 3), (2**63 + 5, 77)),
])
def test_philox_matches_numpy(oracle_lib, ctr, key):
    c = sum(v << (64 * i) for i, v in enumerate(ctr))
    k = key[0] + (key[1] << 64)
    want = np.random.Philox(key=k, counter=(c - 1) % (1 << 256)).random_raw(4)
    got = oracle.philox4x64(np.array(ctr, np.uint64), np.array(key, np.uint64))
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("seed", [0, 1, 2**40 + 3])
def test_site_keys_match_numpy(oracle_lib, seed):
    H, W = 9, 13
    for order in (0, 1):
        for n, b in ((0, 0), (5, 3), (1000, 17)):
            want = e3_conv.site_keys(order, seed, n, b, H, W)
            got = [oracle.site_key(order, seed, n, b, p) for p in range(H * W)]
            np.testing.assert_array_equal(np.array(got, np.uint64), want)
    # keys never tie: the low 12 bits hold 4095 - pos
    ks = e3_conv.site_keys(1, seed, 3, 1, 64, 64)
    assert len(np.unique(ks)) == 64 * 64


CASES = [
    # (name, B, H, W, C, R, shapes, p_dc, per_env, T, variant)
    ("small3x3", 10, 7, 8, 5, 5, ((3, 3), (1, 2), (2, 1)), 0.5, False, 4, "planted"),
    ("dense", 8, 6, 9, 5, 6, ((2, 2), (1, 2), (1, 1)), 0.9, False, 4, "dense"),
    ("perenv", 6, 6, 6, 5, 4, ((3, 3), (2, 1)), 0.5, True, 3, "planted"),
    ("wide", 4, 5, 33, 4, 4, ((1, 2), (2, 3)), 0.7, False, 3, "dense"),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
@pytest.mark.parametrize("order", [0, 1])
@pytest.mark.parametrize("mode", [0, 1])
def test_control_matches_conv_form(oracle_lib, case, order, mode):
    name, B, H, W, C, R, shapes, p_dc, per_env, T, variant = case
    wl = inputs.Workload(name, 200 + len(name), B=B, H=H, W=W, C=C, R=R, shapes=shapes,
                         p_dc=p_dc, per_env=per_env, T=T, L=3)
    for seed in range(2):
        maps, rules, acts = inputs.make_all(wl, seed, variant)
        g = np.random.default_rng(1000 + seed)
        S = B if per_env else 1
        limit, inhibit = random_control(g, S, R)
        control = (limit, inhibit, order, 12345 + seed)
        got = oracle.run(wl, maps, rules, acts, rule_mode=mode, control=control)
        want = e3_conv.run(maps, rules, acts, L=wl.L, per_env=per_env, sequential=bool(mode),
                           control=control)
        for a, b_, what in zip(got, want, ("maps", "rewards", "done")):
            np.testing.assert_array_equal(a, b_, err_msg=f"{name} seed {seed} {what}")
        # the control changed something in at least one case of the set
        plain = oracle.run(wl, maps, rules, acts, rule_mode=mode)
        if name in ("dense", "small3x3"):
            assert not all(np.array_equal(x, y) for x, y in zip(got, plain))


def test_limits_that_never_bind_change_nothing(oracle_lib):
    wl = inputs.Workload("nb", 5, B=8, H=6, W=7, C=5, R=5, shapes=((2, 2), (1, 3)), p_dc=0.8,
                         per_env=False, T=4)
    maps, rules, acts = inputs.make_all(wl, 0, "dense")
    plain = oracle.run(wl, maps, rules, acts)
    big = np.full((1, wl.R), wl.H * wl.W, np.int32)
    for order in (0, 1):
        got = oracle.run(wl, maps, rules, acts, control=(big, None, order, 9))
        assert all(np.array_equal(x, y) for x, y in zip(got, plain))


@pytest.mark.parametrize("K", [1, 2, 5, 17])
@pytest.mark.parametrize("order", [0, 1])
def test_everywhere_rule_applies_exactly_K_times(oracle_lib, K, order):
    # one 1x1 rule with an all-don't-care input (matches at every anchor) that sets tile 4;
    # limited to K it sets exactly K cells and pays K; row-major order picks the first K
    B, H, W, C = 3, 5, 6, 5
    o = oracle.Oracle(B, H, W, C, 1, 1, 1, False, 0)
    ip = np.full((1, 1, C + 1, 1, 1), -1, np.int8)
    op = np.full((1, 1, C + 1, 1, 1), -1, np.int8)
    op[0, 0, 4, 0, 0] = 1
    o.load_rules(np.array([[[1, 1]]], np.int32), ip, op, np.array([[1]], np.int32))
    o.set_rule_control(np.array([[K]], np.int32), None, order, 31)
    maps = np.zeros((B, C, H, W), np.uint8)
    maps[:, P, 2, 3] = 1
    o.reset(maps)
    r, d = o.step(np.zeros(B, np.uint8))
    got = o.maps()[:, 4].reshape(B, -1)
    assert (got.sum(1) == K).all() and (r == K).all() and not d.any()
    if order == 0:
        assert (got[:, :K] == 1).all()
    else:
        for b in range(B):
            keys = e3_conv.site_keys(1, 31, 0, b, H, W)
            np.testing.assert_array_equal(np.sort(np.nonzero(got[b])[0]),
                                          np.sort(np.argsort(-keys.astype(np.float64))[:K]))
    o.close()


def test_random_order_changes_with_step_and_env(oracle_lib):
    # the random channel is drawn per batch step and per env: a once-per-step rule that
    # matches everywhere picks different cells over steps and across envs
    B, H, W, C = 4, 8, 8, 5
    o = oracle.Oracle(B, H, W, C, 1, 1, 1, False, 0)
    ip = np.full((1, 1, C + 1, 1, 1), -1, np.int8)
    op = np.full((1, 1, C + 1, 1, 1), -1, np.int8)
    op[0, 0, 4, 0, 0] = 1
    o.load_rules(np.array([[[1, 1]]], np.int32), ip, op, np.array([[0]], np.int32))
    o.set_rule_control(np.array([[1]], np.int32), None, 1, 5)
    maps = np.zeros((B, C, H, W), np.uint8)
    maps[:, P, 0, 0] = 1
    o.reset(maps)
    picks = []
    for _ in range(6):
        before = o.maps()[:, 4].reshape(B, -1).copy()
        o.step(np.zeros(B, np.uint8))
        after = o.maps()[:, 4].reshape(B, -1)
        new = after & (1 - before)
        picks.append([int(np.nonzero(new[b])[0][0]) if new[b].any() else -1 for b in range(B)])
    picks = np.array(picks)
    assert len(set(picks[:, 0].tolist())) > 1
    assert len(set(picks[0].tolist())) > 1
    o.close()


def test_control_validation(oracle_lib):
    o = oracle.Oracle(2, 4, 4, 4, 3, 1, 1, True, 0)
    with pytest.raises(oracle.OracleError) as e:
        o.set_rule_control(None, None, 0, 0)          # before load_rules
    assert e.value.code == oracle.AVO_ESTATE
    ip = np.full((2, 3, 5, 1, 1), -1, np.int8)
    o.load_rules(np.ones((2, 3, 2), np.int32), ip, ip, np.zeros((2, 3), np.int32))
    o.set_rule_control(np.zeros((2, 3), np.int32), np.zeros((2, 3, 3), np.uint8), 1, 7)
    bad_lim = np.zeros((2, 3), np.int32)
    bad_lim[1, 2] = -1
    inh_self = np.zeros((2, 3, 3), np.uint8)
    inh_self[0, 1, 1] = 1
    inh_back = np.zeros((2, 3, 3), np.uint8)
    inh_back[1, 2, 0] = 1
    for args in ((bad_lim, None, 0, 0), (None, inh_self, 0, 0), (None, inh_back, 0, 0),
                 (None, None, 2, 0)):
        with pytest.raises(oracle.OracleError) as e:
            o.set_rule_control(*args)
        assert e.value.code == oracle.AVO_EINVAL
    o.close()


# Planted mistakes in the control code; each must fail the control fixtures or the
# convolution-form cross-check.
MUTANTS = {
    "overlap_rows_short": ("by < ay + n && ay < by + nq", "by + 1 < ay + n && ay < by + nq"),
    "overlap_cols_short": ("bx < ax + m && ax < bx + mq", "bx < ax + m && ax + 1 < bx + mq"),
    "order_reversed": ("uint32_t rank = (uint32_t)(4095 - pos);", "uint32_t rank = (uint32_t)pos;"),
    "limit_off_by_one": ("uint32_t cut = keys[lim - 1];", "uint32_t cut = keys[lim];"),
    "random_word_high_half_only": ("out[w / 2] >> (32 * (w % 2))", "out[w / 2] >> 32"),
    "step_number_frozen": ("    ab->step_no += 1;\n", ""),
    "env_not_in_counter": ("avo_random_word(seed, n, (uint64_t)b, 0, (uint64_t)pos)",
                           "avo_random_word(seed, n, 0, 0, (uint64_t)pos)"),
    "keys_sorted_ascending": ("return x < y ? 1 : (x > y ? -1 : 0);",
                              "return x < y ? -1 : (x > y ? 1 : 0);"),
    "moves_limited_too": ("const int lim = (loaded && ab->limit)", "const int lim = (ab->limit)"),
    "inhibition_ignored": ("if (hit && loaded && ab->inhibit &&", "if (hit && loaded && 0 &&"),
}


def pin_control_fixtures(lib):
    for path in fixtures.all_fixtures():
        fx = fixtures.parse(path)
        if not fx.has_control:
            continue
        shape, ip, op, rw, mh, mw = fx.abi_rules()
        o = oracle.Oracle(1, fx.H, fx.W, fx.C, len(fx.rules), mh, mw, False, fx.L,
                          lib_path=lib, rule_mode=fx.mode)
        o.load_rules(shape, ip, op, rw)
        o.set_rule_control(*fx.abi_control())
        o.reset(fx.init[None])
        for st in fx.steps:
            r, d = o.step(np.array([st.action], np.uint8))
            if not (np.array_equal(o.maps()[0], st.after) and r[0] == st.reward
                    and d[0] == st.done):
                o.close()
                return False
        o.close()
    return True


def pin_control_conv(lib):
    for case in CASES[:3]:
        name, B, H, W, C, R, shapes, p_dc, per_env, T, variant = case
        wl = inputs.Workload(name, 200 + len(name), B=B, H=H, W=W, C=C, R=R, shapes=shapes,
                             p_dc=p_dc, per_env=per_env, T=T, L=3)
        maps, rules, acts = inputs.make_all(wl, 0, variant)
        S = B if per_env else 1
        limit, inhibit = random_control(np.random.default_rng(1000), S, R)
        for order in (0, 1):
            control = (limit, inhibit, order, 12345)
            got = oracle.run(wl, maps, rules, acts, lib_path=lib, control=control)
            want = e3_conv.run(maps, rules, acts, L=wl.L, per_env=per_env, control=control)
            if not all(np.array_equal(a, b) for a, b in zip(got, want)):
                return False
    return True


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    return tmp_path_factory.mktemp("control_mutants")


def test_unmutated_oracle_passes_control_pins(oracle_lib):
    assert pin_control_fixtures(oracle.LIB)
    assert pin_control_conv(oracle.LIB)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_control_mutant_is_caught(oracle_lib, mutant_dir, name):
    old, new = MUTANTS[name]
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/found"
    path = os.path.join(str(mutant_dir), f"avo_{name}.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib = oracle.build(out=os.path.join(str(mutant_dir), f"libavo_{name}.so"), src=path,
                       extra=("-I", oracle.HERE))
    assert not (pin_control_fixtures(lib) and pin_control_conv(lib)), \
        f"mutant {name} passes every control pin"
