"""GPU vs oracle on the limits and degenerate cases: the most channels, a pattern as large
as the map, one-row and one-column maps, rules with no specified input entry, many rules,
no loaded rules, a single environment, 33- and 64-wide maps, out-of-range action values.
Maps, rewards and done flags are compared after every step."""
import numpy as np
import pytest

import oracle
from gpu_util import first_mismatch, gpu_run, group_ok, require_gpu, rows_ok, say
from paper_2407_04221_amd import inputs

pytestmark = pytest.mark.gpu


def W_(name, cid, **kw):
    base = dict(per_env=False, T=12, L=5, p_dc=0.5)
    base.update(kw)
    return inputs.Workload(name, cid, **base)


CASES = {
    "channels31": W_("channels31", 41, B=37, H=16, W=16, C=31, R=10, shapes=((4, 4), (1, 1))),
    "pattern_is_map": W_("pattern_is_map", 42, B=21, H=16, W=16, C=8, R=2, shapes=((16, 16),)),
    "pattern_is_map8": W_("pattern_is_map8", 43, B=9, H=8, W=8, C=4, R=3, shapes=((8, 8), (8, 1))),
    "one_row": W_("one_row", 44, B=19, H=1, W=16, C=5, R=4, shapes=((1, 1), (1, 3))),
    "one_col": W_("one_col", 45, B=19, H=16, W=1, C=5, R=4, shapes=((1, 1), (3, 1))),
    "many_rules": W_("many_rules", 46, B=30, H=16, W=16, C=6, R=60, shapes=((3, 3), (2, 5)),
                     T=6),
    "one_env": W_("one_env", 47, B=1, H=11, W=7, C=4, R=5, shapes=((2, 2), (1, 3))),
    "wide33": W_("wide33", 48, B=6, H=33, W=33, C=6, R=6, shapes=((3, 3), (1, 4)), T=8),
    "big64": W_("big64", 49, B=3, H=64, W=64, C=20, R=40, shapes=((5, 5), (2, 3)), T=4),
    "per_env_small": W_("per_env_small", 50, B=13, H=10, W=12, C=5, R=5,
                        shapes=((3, 3), (1, 2)), per_env=True),
    "max_rules": W_("max_rules", 55, B=5, H=8, W=8, C=4, R=252, shapes=((1, 1), (2, 2)), T=4),
    # maps above 32 rows: the rows engine's four-wave variant, with 4-byte rows and with
    # per-environment rule sets
    "tall40x20": W_("tall40x20", 56, B=7, H=40, W=20, C=6, R=12, shapes=((3, 3), (2, 1)), T=10),
    "tall_per_env": W_("tall_per_env", 57, B=5, H=48, W=40, C=5, R=8,
                       shapes=((3, 3), (1, 2)), per_env=True, T=10),
    # two rows a lane on a map of 24 rows (second rows 24..31 of each group empty), patterns
    # up to 4 x 4 (three pad rows under the planes), per-environment rules
    "mid24x20": W_("mid24x20", 59, B=11, H=24, W=20, C=7, R=9,
                   shapes=((4, 4), (1, 3), (2, 1)), per_env=True, T=14),
    # patterns wider than 8 columns (the group engine tests a plane row in blocks of 8)
    "wide_pat": W_("wide_pat", 60, B=9, H=12, W=24, C=5, R=3, shapes=((1, 13), (2, 9)),
                   per_env=True, T=14),
}
LANE16 = {n for n, w in CASES.items() if w.H <= 16 and w.W <= 16 and not w.per_env}


def engines(name):
    wl = CASES[name]
    out = ["generic", "lane16"] if name in LANE16 else ["generic"]
    # the wave engine: C + 1 planes of H + 16 rows, one 80-row match plane per rule, two
    # 64-row vote accumulators per plane (4-byte rows for W <= 32, else 8), a word per rule
    # and three 64-word step blocks within 64 KiB
    rowb, rt = (4 if wl.W <= 32 else 8), wl.R + 4
    if ((wl.C + 1) * (wl.H + 16) + rt * 80 + 2 * (wl.C + 1) * 64) * rowb + 4 * (rt + 2 + 192) <= 65536:
        out.append("wave")
    return out + (["rows"] if rows_ok(wl) else []) + (["group"] if group_ok(wl) else [])


def check(wl, maps, rules, actions, engine):
    want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8)
    seq, final, r, d, eng = gpu_run(wl, maps, rules, actions, engine=engine, mode="step")
    for t in range(actions.shape[0]):
        assert first_mismatch(seq[t], want_m[t]) is None, \
            f"maps differ at step {t}, index {first_mismatch(seq[t], want_m[t])}"
        np.testing.assert_array_equal(r[t], want_r[t], err_msg=f"rewards, step {t}")
        np.testing.assert_array_equal(d[t], want_d[t], err_msg=f"done, step {t}")
    return want_r


@pytest.mark.parametrize("variant", ["literal", "planted", "dense"])
@pytest.mark.parametrize("name,engine", [(n, e) for n in sorted(CASES) for e in engines(n)])
def test_edge_case(name, engine, variant):
    require_gpu()
    wl = CASES[name]
    say(f"[edge] {name} engine={engine} variant={variant}")
    maps, rules, actions = inputs.make_all(wl, 0, variant)
    check(wl, maps, rules, actions, engine)


@pytest.mark.parametrize("variant", ["planted", "dense"])
@pytest.mark.parametrize("name", ["tall40x20", "tall_per_env", "wide33", "c5", "c5_per_env"])
def test_tall_maps_in_long_launches(name, variant):
    """Rows engine on maps above 32 rows in launches of 20 steps (the rule program staged in
    LDS, four waves per environment sharing the probe, the filter and the matching)."""
    require_gpu()
    if name.startswith("c5"):
        wl = inputs.WORKLOADS["c5"].with_(B=3, T=40, L=5, per_env=name == "c5_per_env")
    else:
        wl = CASES[name].with_(T=40)
    if not rows_ok(wl):
        pytest.skip("not eligible for the rows engine")
    say(f"[tall step_n] {name} variant={variant}")
    maps, rules, actions = inputs.make_all(wl, 3, variant)
    want_m, want_r, want_d = oracle.run(wl, maps, rules, actions, nthreads=8)
    _, final, r, d, eng = gpu_run(wl, maps, rules, actions, engine="rows", mode="step_n",
                                  chunk=20)
    np.testing.assert_array_equal(r, want_r)
    np.testing.assert_array_equal(d, want_d)
    np.testing.assert_array_equal(final, want_m[-1])


@pytest.mark.parametrize("engine", ["generic", "lane16", "wave", "rows", "group"])
def test_rules_with_no_specified_input(engine):
    """An all-don't-care input matches at every anchor (the paper's empty "no-op" rules,
    Sec. 2.2.1); with outputs it writes everywhere, with heavily overlapping votes."""
    require_gpu()
    wl = W_("dc", 51, B=17, H=9, W=14, C=5, R=3, shapes=((2, 3), (1, 1), (3, 2)), T=6)
    maps, (shape, ip, op, rw), actions = inputs.make_all(wl, 0, "dense")
    ip[:] = -1
    op[:, 1] = -1                 # rule 1 matches everywhere and changes nothing
    rw[:] = (1, 1, -1)
    r = check(wl, maps, (shape, ip, op, rw), actions, engine)
    assert (r != 0).all()


@pytest.mark.parametrize("engine", ["generic", "lane16", "wave", "rows", "group"])
def test_no_loaded_rules(engine):
    require_gpu()
    wl = W_("moves", 52, B=41, H=13, W=16, C=4, R=0, shapes=((1, 1),), T=30, L=0)
    maps = inputs.make_maps(wl, 0)
    actions = inputs.make_actions(wl, 0)
    empty = (np.zeros((1, 0, 2), np.int32), np.zeros((1, 0, 5, 1, 1), np.int8),
             np.zeros((1, 0, 5, 1, 1), np.int8), np.zeros((1, 0), np.int32))
    check(wl, maps, empty, actions, engine)


@pytest.mark.parametrize("engine", ["generic", "lane16", "wave", "rows", "group"])
def test_out_of_range_actions_are_no_ops(engine):
    require_gpu()
    wl = W_("acts", 53, B=24, H=8, W=8, C=4, R=2, shapes=((1, 2),), T=10)
    maps, rules, _ = inputs.make_all(wl, 0, "planted")
    actions = np.random.default_rng(5).integers(0, 256, size=(wl.T, wl.B)).astype(np.uint8)
    actions[:, ::3] = 0
    check(wl, maps, rules, actions, engine)


@pytest.mark.parametrize("engine", ["rows", "wave", "generic"])
def test_vote_counts_beyond_4096(engine):
    """16 all-don't-care 16 x 16 rules vote +1 and 15 vote -1 on the goal plane of a 64 x 64
    map: a cell away from the edges is covered by 256 anchors of each rule, so it gets
    4096 plus and 3840 minus votes (plus its old value), and the exact counts need more than
    12 bits (a 12-bit count of the plus votes would wrap to 0 and clear the cell)."""
    require_gpu()
    R = 31
    wl = W_("votes", 54, B=2, H=64, W=64, C=4, R=R, shapes=((16, 16),), T=2, L=0)
    maps, (shape, ip, op, rw), actions = inputs.make_all(wl, 0, "literal")
    ip[:] = -1
    op[:] = -1
    op[:, :16, 3] = 1
    op[:, 16:, 3] = 0
    rw[:] = 0
    actions[:] = 0
    want_m, want_r, want_d = oracle.run(wl, maps, (shape, ip, op, rw), actions, nthreads=8)
    assert want_m[0][:, 3, 15:49, 15:49].all()      # the interior became (or stayed) goal
    check(wl, maps, (shape, ip, op, rw), actions, engine)


@pytest.mark.parametrize("shape", [(3, 3), (1, 3), (1, 7)])
@pytest.mark.parametrize("rules_per_sign", [1, 2])
@pytest.mark.parametrize("engine", ["group", "wave", "generic"])
def test_overlapping_votes_of_both_signs(engine, rules_per_sign, shape):
    """All-don't-care n x m rules, half voting +1 and half -1 on the goal plane: a cell away
    from the edges gets n m votes of each sign per rule, so every cell needs an exact count.
    The rules' vote entries on the plane number 6 (1 x 3, one rule per sign), 12, 14 (1 x 7:
    counts up to 15, the most 4-bit counters hold), 18, 28 and 36 (beyond 4 bits)."""
    require_gpu()
    R = 2 * rules_per_sign
    wl = W_("both", 58, B=7, H=12, W=15, C=5, R=R, shapes=(shape,), T=4, L=0)
    maps, (shape, ip, op, rw), actions = inputs.make_all(wl, 0, "literal")
    ip[:] = -1
    op[:] = -1
    op[:, :rules_per_sign, 3] = 1
    op[:, rules_per_sign:, 3] = 0
    rw[:] = 0
    check(wl, maps, (shape, ip, op, rw), actions, engine)
