"""Oracle search (oracle/search.py: level-synchronous search with state deduplication that
keeps the higher-reward, then shallower node, paper Sec. 2.2.1) pinned by:

  * a hand-worked corridor: per-level counts, the best reward and the visit at which it is
    first found, with and without an episode length that makes level-3 children terminal;
  * brute force with the convolution-form stepper (tests/e3_conv.py, independent of the
    oracle): with zero rewards the level-d frontier is exactly the set of states whose
    shortest action sequence has length d; with rewards the best reward after D levels is
    the maximum over every action sequence of length <= D and its prefixes;
  * budget and frontier cuts, and planted mistakes in the search that these pins catch.
"""
import importlib.util
import itertools
import os

import numpy as np
import pytest

import e3_conv
import oracle
from oracle import search as osearch
from paper_2407_04221_amd import inputs

E, WALL, P, G = 0, 1, 2, 3


def corridor(L=100):
    C = 4
    root = np.zeros((C, 1, 4), np.uint8)
    root[P, 0, 0] = 1
    root[G, 0, 3] = 1
    shape = np.array([[[1, 2]]], np.int32)
    ip = np.full((1, 1, C + 1, 1, 2), -1, np.int8)
    op = np.full((1, 1, C + 1, 1, 2), -1, np.int8)
    ip[0, 0, P, 0, 0] = 1                 # food: the player moves onto the goal and eats it
    ip[0, 0, C, 0, 1] = 1
    ip[0, 0, G, 0, 1] = 1
    op[0, 0, P, 0, 0] = 0
    op[0, 0, P, 0, 1] = 1
    op[0, 0, C, 0, 1] = 0
    op[0, 0, G, 0, 1] = 0
    rules = (shape, ip, op, np.array([[1]], np.int32))
    return root, rules, L


def test_corridor_worked_case(oracle_lib):
    # P . . G: only "right" makes progress; level 3 eats the goal (visit 10 + 1 + 2 = 13);
    # then the player can walk back left one new cell per level until the wall of the map
    root, rules, L = corridor()
    s = osearch.Search(1, 4, 4, rules, L)
    levels = s.run(root, budget=10**6)
    assert [lv["children"] for lv in levels] == [5] * 7
    assert [lv["survivors"] for lv in levels] == [1, 1, 1, 1, 1, 1, 0]
    assert [lv["terminal"] for lv in levels] == [0] * 7
    assert levels[-1]["visited"] == 35
    assert (levels[-1]["best_reward"], levels[-1]["best_visit"]) == (1, 13)
    # with episodes of 3 steps every level-3 child is terminal, but the reward still counts
    s = osearch.Search(1, 4, 4, rules, 3)
    levels = s.run(root, budget=10**6)
    assert [lv["survivors"] for lv in levels] == [1, 1, 0]
    assert [lv["terminal"] for lv in levels] == [0, 0, 5]
    assert (levels[-1]["best_reward"], levels[-1]["best_visit"]) == (1, 13)


def brute_force(root, rules_list, D, actions):
    """Every action sequence of length <= D, stepped with the conv form (all sequences of one
    length as one batch); a sequence stops when its episode ends (no player left).  Returns
    (first depth of every non-terminal state, best reward over all sequences and prefixes)."""
    first = {root.tobytes(): 0}
    best = 0
    maps = root[None].copy()                  # live sequences of the current length
    totals = np.zeros(1, np.int64)
    for length in range(1, D + 1):
        if len(maps) == 0:
            break
        A = len(actions)
        maps = np.repeat(maps, A, axis=0)
        totals = np.repeat(totals, A)
        acts = np.tile(np.array(list(actions)), len(maps) // A)
        maps, rho = e3_conv.step(maps, rules_list, acts)
        totals = totals + rho.astype(np.int64)
        if len(totals):
            best = max(best, int(totals.max()))
        alive = maps[:, P].reshape(len(maps), -1).sum(1) > 0
        maps, totals = maps[alive], totals[alive]
        for m in maps:
            first.setdefault(m.tobytes(), length)
    return first, best


@pytest.mark.parametrize("seed", range(4))
def test_zero_reward_levels_are_shortest_distances(oracle_lib, seed):
    wl = inputs.Workload("s", 600 + seed, B=1, H=3, W=4, C=5, R=3, shapes=((1, 2), (2, 1)),
                         p_dc=0.6, per_env=False, T=1)
    maps, (shape, ip, op, rw), _ = inputs.make_all(wl, seed, "planted")
    rw = np.zeros_like(rw)
    D = 4
    first, _ = brute_force(maps[0], e3_conv.rules_from_abi(shape, ip, op, rw), D, range(5))
    s = osearch.Search(3, 4, 5, (shape, ip, op, rw), 100)
    s.begin(maps[0])
    for d in range(1, D + 1):
        s.expand(10**9)
        got = {m.tobytes() for m in s.frontier_arrays()[0]}
        want = {k for k, v in first.items() if v == d}
        assert got == want, f"level {d}"


@pytest.mark.parametrize("seed", range(4))
def test_best_reward_is_the_brute_force_maximum(oracle_lib, seed):
    wl = inputs.Workload("s", 700 + seed, B=1, H=3, W=4, C=5, R=4, shapes=((1, 2), (1, 1)),
                         p_dc=0.6, per_env=False, T=1)
    maps, rules, _ = inputs.make_all(wl, seed, "dense")
    D = 4
    _, best = brute_force(maps[0], e3_conv.rules_from_abi(*rules), D, range(5))
    s = osearch.Search(3, 4, 5, rules, 100)
    levels = s.run(maps[0], budget=10**9, max_levels=D)
    assert levels[-1]["best_reward"] == best


def test_budget_and_frontier_cuts(oracle_lib):
    root, rules, L = corridor()
    root = np.zeros((4, 3, 3), np.uint8)
    root[P, 1, 1] = 1
    s = osearch.Search(3, 3, 4, rules, 100, max_frontier=2)
    s.begin(root)
    lv = s.expand(10**6)
    assert lv["children"] == 5 and lv["survivors"] == 4 and lv["frontier"] == 2
    lv = s.expand(7)                          # 2 parents x 5 actions, cut to 7
    assert lv["children"] == 7 and lv["visited"] == 12
    kept = s.frontier_arrays()
    lv = s.expand(0)                          # nothing expanded, frontier kept
    assert lv["children"] == 0
    np.testing.assert_array_equal(s.frontier_arrays()[0], kept[0])
    # four actions (no no-op)
    s4 = osearch.Search(3, 3, 4, rules, 100, num_actions=4)
    s4.begin(root)
    assert s4.expand(10**6)["children"] == 4


MUTANTS = {
    "prefers_deeper": ("val = (reward, -depth)", "val = (reward, depth)"),
    "ties_keep_last": ("val > best_in_level[key][0]", "val >= best_in_level[key][0]"),
    "terminal_expanded": ('                info["terminal"] += 1\n                continue\n',
                          '                info["terminal"] += 1\n'),
    "visit_off_by_one": ("visit = self.visited + 1 + i", "visit = self.visited + i"),
    "counter_not_set": ("        o.set_counters(", "        (lambda *_: None)("),
    "best_not_strict": ("if reward > self.best[0]:", "if reward >= self.best[0]:"),
    "reward_not_accumulated": ("reward = self.frontier[p][1] + int(r[i])", "reward = int(r[i])"),
}


def load_mutant(name, tmpdir):
    old, new = MUTANTS[name]
    src = open(osearch.__file__).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/found"
    path = os.path.join(tmpdir, f"search_{name}.py")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    spec = importlib.util.spec_from_file_location(f"search_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def pins(mod):
    root, rules, _ = corridor()
    for L, want in ((100, ([1, 1, 1, 1, 1, 1, 0], 35, (1, 13))), (3, ([1, 1, 0], 15, (1, 13)))):
        levels = mod.Search(1, 4, 4, rules, L).run(root, budget=10**6)
        if ([lv["survivors"] for lv in levels], levels[-1]["visited"],
                (levels[-1]["best_reward"], levels[-1]["best_visit"])) != want:
            return False
    # rewards accumulate along the path: P . G G eats two goals
    root2 = root.copy()
    root2[G, 0, 2] = 1
    levels = mod.Search(1, 4, 4, rules, 100).run(root2, budget=10**6)
    if levels[-1]["best_reward"] != 2:
        return False
    # ties inside a level: on a 3 x 3 map with the player in the centre, level 2 reaches each
    # corner from two level-1 parents at the same depth and reward; the lower child index is
    # kept (children 2, 4, 8, 14 rather than 6, 16, 12, 18), which fixes the frontier order
    # (0,2), (0,0), (2,2), (2,0); keeping the later copies would give (0,2), (2,2), (0,0), (2,0)
    C = 4
    rules0 = (np.zeros((1, 0, 2), np.int32), np.zeros((1, 0, C + 1, 1, 1), np.int8),
              np.zeros((1, 0, C + 1, 1, 1), np.int8), np.zeros((1, 0), np.int32))
    centre = np.zeros((C, 3, 3), np.uint8)
    centre[P, 1, 1] = 1
    s = mod.Search(3, 3, C, rules0, 100)
    s.begin(centre)
    s.expand(10**6)
    s.expand(10**6)
    order = [tuple(np.argwhere(m[P])[0]) for m in s.frontier_arrays()[0]]
    if order != [(0, 2), (0, 0), (2, 2), (2, 0)]:
        return False
    # a deeper copy of a state with the same reward must be pruned
    s3 = mod.Search(1, 4, 4, rules, 100)
    s3.begin(root)
    s3.expand(10**6)
    if s3.expand(10**6)["survivors"] != 1:
        return False
    return True


def test_unmutated_search_passes_pins(oracle_lib):
    assert pins(osearch)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_search_mutant_is_caught(oracle_lib, tmp_path, name):
    mod = load_mutant(name, str(tmp_path))
    assert not pins(mod), f"mutant {name} passes every search pin"
