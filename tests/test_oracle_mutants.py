"""The oracle's pins are strong enough to catch plausible mistakes.

Each mutant is a copy of oracle/avo.c with one planted mistake (a sign, an index, an
off-by-one, a dropped term, a different reading of rule order), compiled on the CPU to a
temporary library.  Every mutant must fail at least one pin: the worked cases, the
convolution-form cross-check, the exhaustive move check or the order-invariance check.
"""
import os

import numpy as np
import pytest

import e3_conv
import fixtures
import oracle
from paper_2407_04221_amd import inputs

MUTANTS = {
    "force_up_down_swapped": ("{{0, 0}, {-1, 0}, {0, 1}, {1, 0}, {0, -1}}",
                              "{{0, 0}, {1, 0}, {0, 1}, {-1, 0}, {0, -1}}"),
    "force_left_right_swapped": ("{{0, 0}, {-1, 0}, {0, 1}, {1, 0}, {0, -1}}",
                                 "{{0, 0}, {-1, 0}, {0, -1}, {1, 0}, {0, 1}}"),
    "clear_vote_sign": ("return in == 0 ? 0 : -1;", "return in == 0 ? 0 : 1;"),
    "set_vote_ignores_input": ("if (out == 1) return in == 1 ? 0 : 1;", "if (out == 1) return 1;"),
    "anchor_rows_short": ("ay + rv.n <= H", "ay + rv.n < H"),
    "anchor_cols_short": ("ax + rv.m <= W", "ax + rv.m < W"),
    "clamp_threshold": ("(X[k] + delta[k] >= 1) ? 1 : 0;\n\n", "(X[k] + delta[k] > 1) ? 1 : 0;\n\n"),
    "sequential_votes_carried_over": ("                delta[k] = 0;\n", ""),
    "dont_care_read_as_zero": ("if (want == -1) continue;", "if (want == -1) want = 0;"),
    "wall_does_not_block": ("in[k][CH_WALL][ty][tx] = 0;", "(void)0;"),
    "reward_not_accumulated": ("rho += rv.reward;", "rho = rv.reward;"),
    "episode_length_ignored": ("(ab->episode_len > 0 && ab->t[b] == ab->episode_len)", "0"),
    "reset_to_empty_map": ("memcpy(D, ab->init_maps + (size_t)b * C * plane, (size_t)C * plane);",
                           "memset(D, 0, (size_t)C * plane);"),
    "vote_column_dropped": ("delta[(size_t)c * plane + (size_t)(ay + i) * W + ax + j] += k;",
                            "delta[(size_t)c * plane + (size_t)(ay + i) * W + ax] += k;"),
    "rules_applied_in_sequence": (
        "    for (int r = 0; r < nrules; r++) {\n",
        "    for (int r = 0; r < nrules; r++) {\n"
        "        for (size_t q = 0; q < (size_t)C1 * plane; q++) {\n"
        "            X[q] = (X[q] + delta[q] >= 1) ? 1 : 0; delta[q] = 0; }\n"),
}


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    return tmp_path_factory.mktemp("mutants")


def build_mutant(name, outdir):
    old, new = MUTANTS[name]
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/found"
    path = os.path.join(outdir, f"avo_{name}.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    return oracle.build(out=os.path.join(outdir, f"libavo_{name}.so"), src=path,
                        extra=("-I", oracle.HERE))


def pin_worked_cases(lib):
    for path in fixtures.all_fixtures():
        fx = fixtures.parse(path)
        shape, ip, op, rw, mh, mw = fx.abi_rules()
        o = oracle.Oracle(1, fx.H, fx.W, fx.C, max(len(fx.rules), 1), mh, mw, False, fx.L,
                          lib_path=lib, rule_mode=fx.mode)
        o.load_rules(shape, ip, op, rw)
        if fx.has_control:
            o.set_rule_control(*fx.abi_control())
        o.reset(fx.init[None])
        for st in fx.steps:
            r, d = o.step(np.array([st.action], np.uint8))
            if not (np.array_equal(o.maps()[0], st.after) and r[0] == st.reward
                    and d[0] == st.done):
                return False
        o.close()
    return True


def pin_conv_form(lib):
    for seed in range(3):
        for variant in ("literal", "planted", "dense"):
            wl = inputs.Workload("t", 90 + seed, B=12, H=6, W=7, C=5, R=4,
                                 shapes=((3, 3), (2, 1), (1, 2)), p_dc=0.5, per_env=False,
                                 T=4, L=3)
            maps, rules, actions = inputs.make_all(wl, seed, variant)
            want = e3_conv.run(maps, rules, actions, L=wl.L)
            got = oracle.run(wl, maps, rules, actions, lib_path=lib)
            if not all(np.array_equal(a, b) for a, b in zip(got, want)):
                return False
    return True


def pin_moves(lib):
    g = np.random.default_rng(0)
    B = 512
    walls = (g.random((B, 4, 4)) < 0.4).astype(np.uint8)
    o = oracle.Oracle(B, 4, 4, 4, 0, 1, 1, False, 0, lib_path=lib)
    o.load_rules(np.zeros((1, 0, 2), np.int32), np.zeros((1, 0, 5, 1, 1), np.int8),
                 np.zeros((1, 0, 5, 1, 1), np.int8), np.zeros((1, 0), np.int32))
    dirs = {0: (0, 0), 1: (-1, 0), 2: (0, 1), 3: (1, 0), 4: (0, -1)}
    ok = True
    for py, px in ((0, 0), (1, 2), (3, 3)):
        maps = np.zeros((B, 4, 4, 4), np.uint8)
        maps[:, 1] = walls
        maps[:, 2, py, px] = 1
        for a, (dy, dx) in dirs.items():
            o.reset(maps)
            o.step(np.full(B, a, np.uint8))
            want = maps.copy()
            ty, tx = py + dy, px + dx
            if a and 0 <= ty < 4 and 0 <= tx < 4:
                free = walls[:, ty, tx] == 0
                want[free, 2, py, px] = 0
                want[free, 2, ty, tx] = 1
            ok &= np.array_equal(o.maps(), want)
    o.close()
    return ok


def pin_order_invariance(lib):
    wl = inputs.Workload("t", 77, B=16, H=7, W=8, C=5, R=6, shapes=((3, 3), (1, 2), (2, 2)),
                         p_dc=0.55, per_env=False, T=2)
    maps, (shape, ip, op, rw), acts = inputs.make_all(wl, 1, "planted")
    perm = np.arange(wl.R)[::-1].copy()
    a = oracle.run(wl, maps, (shape, ip, op, rw), acts, lib_path=lib)
    b = oracle.run(wl, maps, (shape[:, perm], ip[:, perm], op[:, perm], rw[:, perm]), acts,
                   lib_path=lib)
    return all(np.array_equal(x, y) for x, y in zip(a, b))


PINS = (pin_worked_cases, pin_conv_form, pin_moves, pin_order_invariance)


def test_unmutated_oracle_passes_every_pin(oracle_lib):
    for pin in PINS:
        assert pin(oracle.LIB), pin.__name__


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(oracle_lib, mutant_dir, name):
    lib = build_mutant(name, str(mutant_dir))
    caught = [pin.__name__ for pin in PINS if not pin(lib)]
    assert caught, f"mutant {name} passes every pin"
