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
    "reward_not_accumulated": ("return [(maps[i], parents[p][1] + int(r[i])",
                               "return [(maps[i], int(r[i])"),
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


# ---------------------------------------------------------------------------------------
# Batched best-first search (oracle/search.py BestFirst)

def two_goals():
    # 3 x 3, player at (1, 0), goals at (1, 1) and (1, 2); the corridor's rule pays 1 when
    # the player moves right onto a goal
    _, rules, _ = corridor()
    root = np.zeros((4, 3, 3), np.uint8)
    root[P, 1, 0] = 1
    root[G, 1, 1] = 1
    root[G, 1, 2] = 1
    return root, rules


def test_best_first_worked_case(oracle_lib):
    # Iteration 1 expands the root: up (visit 2), right (visit 3, eats a goal: reward 1) and
    # down (visit 4) are new.  Best-first then expands the reward-1 node first: its right
    # child (visit 6 + 2 = 8) eats the second goal.  Breadth-first reaches it only at visit
    # 13 (the up node's children come first).
    root, rules = two_goals()
    bf = osearch.BestFirst(3, 3, 4, rules, 100, k=1)
    levels = bf.run(root, budget=10**6, max_levels=2)
    assert [lv["survivors"] for lv in levels] == [3, 4]
    assert (levels[-1]["best_reward"], levels[-1]["best_visit"], levels[-1]["visited"]) == (2, 8, 10)
    assert levels[-1]["frontier"] == 6
    bfs = osearch.Search(3, 3, 4, rules, 100)
    levels = bfs.run(root, budget=10**6, max_levels=2)
    assert (levels[-1]["best_reward"], levels[-1]["best_visit"]) == (2, 13)


def textbook_best_first(root, rules_list, L, budget, actions=range(5)):
    """Plain best-first search with a binary heap and lazy deletion, stepping with the
    convolution form (tests/e3_conv.py); one node expanded per pop."""
    import heapq
    nodes = [(root, 0, 0)]
    best_of = {root.tobytes(): (0, 0)}
    heap = [(0, 0, 0)]                       # (-reward, depth, id)
    visited, best = 0, (0, 0)
    expanded = []
    while heap and visited < budget:
        _, _, nid = heapq.heappop(heap)
        m, rew, dep = nodes[nid]
        if best_of[m.tobytes()] != (rew, -dep):
            continue                         # pruned by a better copy of its state
        expanded.append((m.tobytes(), rew, dep))
        acts = list(actions)[:budget - visited]
        kids, rho = e3_conv.step(np.repeat(m[None], len(acts), 0), rules_list, np.array(acts))
        cand = {}
        for i in range(len(acts)):
            visited += 1
            r = rew + int(rho[i])
            if r > best[0]:
                best = (r, visited)
            done = kids[i, P].sum() == 0 or (L > 0 and dep + 1 == L)
            if done:
                continue
            key = kids[i].tobytes()
            v = (r, -(dep + 1))
            if key not in cand or v > cand[key][0]:
                cand[key] = (v, i)
        for key, (v, i) in sorted(cand.items(), key=lambda kv: kv[1][1]):
            if key not in best_of or v > best_of[key]:
                best_of[key] = v
                nodes.append((kids[i], v[0], -v[1]))
                heapq.heappush(heap, (-v[0], -v[1], len(nodes) - 1))
    return visited, best, expanded


def bf_expanded(bf):
    return [(bf.nodes[i][0].tobytes(), bf.nodes[i][1], bf.nodes[i][2]) for i in bf.expanded]


@pytest.mark.parametrize("seed", range(4))
def test_best_first_k1_is_textbook_best_first(oracle_lib, seed):
    wl = inputs.Workload("s", 800 + seed, B=1, H=3, W=4, C=5, R=3, shapes=((1, 2), (1, 1)),
                         p_dc=0.6, per_env=False, T=1)
    maps, rules, _ = inputs.make_all(wl, seed, "dense")
    for budget in (7, 60, 400):
        want = textbook_best_first(maps[0], e3_conv.rules_from_abi(*rules), 6, budget)
        bf = osearch.BestFirst(3, 4, 5, rules, 6, k=1)
        levels = bf.run(maps[0], budget)
        got = (levels[-1]["visited"], (levels[-1]["best_reward"], levels[-1]["best_visit"]),
               bf_expanded(bf))
        assert got[:2] == want[:2], (budget, got[:2], want[:2])
        assert got[2] == want[2], f"budget {budget}: expansion order differs"


@pytest.mark.parametrize("k", [1, 3, 16])
@pytest.mark.parametrize("seed", range(3))
def test_best_first_finds_the_brute_force_maximum(oracle_lib, k, seed):
    # episodes of L = 4 steps bound the depth, so an unlimited search sees every state that
    # is not dominated: its best reward is the maximum over all action sequences
    wl = inputs.Workload("s", 900 + seed, B=1, H=3, W=4, C=5, R=4, shapes=((1, 2), (1, 1)),
                         p_dc=0.6, per_env=False, T=1)
    maps, rules, _ = inputs.make_all(wl, seed, "dense")
    _, best = brute_force(maps[0], e3_conv.rules_from_abi(*rules), 4, range(5))
    bf = osearch.BestFirst(3, 4, 5, rules, 4, k=k)
    levels = bf.run(maps[0], budget=10**9)
    assert levels[-1]["best_reward"] == best
    assert levels[-1]["frontier"] == 0


BF_MUTANTS = {
    "deeper_first": ("key=lambda i: (-self.nodes[i][1], self.nodes[i][2], i))\n        popped",
                     "key=lambda i: (-self.nodes[i][1], -self.nodes[i][2], i))\n        popped"),
    "no_liveness_check": ("if self.table[self.nodes[i][0].tobytes()] == (self.nodes[i][1],",
                          "if True or self.table[self.nodes[i][0].tobytes()] == (self.nodes[i][1],"),
    "lowest_reward_first": ("key=lambda i: (-self.nodes[i][1], self.nodes[i][2], i))\n        popped",
                            "key=lambda i: (self.nodes[i][1], self.nodes[i][2], i))\n        popped"),
}


def force_pays():
    # 1 x 3 corridor; a rule with no output pays 1 wherever a force tile lies, so every
    # action that places force earns 1 without changing the map: a state is re-reached with a
    # higher reward all the time, and the earlier open copy must then be skipped
    C = 4
    root = np.zeros((C, 1, 3), np.uint8)
    root[P, 0, 0] = 1
    ip = np.full((1, 1, C + 1, 1, 1), -1, np.int8)
    op = np.full((1, 1, C + 1, 1, 1), -1, np.int8)
    ip[0, 0, C, 0, 0] = 1
    rules = (np.array([[[1, 1]]], np.int32), ip, op, np.array([[1]], np.int32))
    return root, rules


def test_best_first_skips_dominated_open_nodes(oracle_lib):
    root, rules = force_pays()
    for budget in (30, 200):
        want = textbook_best_first(root, e3_conv.rules_from_abi(*rules), 5, budget)
        bf = osearch.BestFirst(1, 3, 4, rules, 5, k=1)
        levels = bf.run(root, budget)
        assert (levels[-1]["visited"], (levels[-1]["best_reward"], levels[-1]["best_visit"]),
                bf_expanded(bf)) == want
        if budget == 200:                                   # the search runs to the end
            assert any(lv["parents"] == 0 for lv in levels)  # and pops a dominated node


def bf_pins(mod):
    root, rules = force_pays()
    want = textbook_best_first(root, e3_conv.rules_from_abi(*rules), 5, 200)
    bf = mod.BestFirst(1, 3, 4, rules, 5, k=1)
    levels = bf.run(root, 200)
    if (levels[-1]["visited"], (levels[-1]["best_reward"], levels[-1]["best_visit"]),
            bf_expanded(bf)) != want:
        return False
    for seed, variant in ((1, "planted"), (25, "dense")):
        wl = inputs.Workload("s", 950 + seed, B=1, H=3, W=4, C=5, R=4,
                             shapes=((1, 2), (1, 1), (2, 1)), p_dc=0.6, per_env=False, T=1)
        maps, rules, _ = inputs.make_all(wl, seed, variant)
        want = textbook_best_first(maps[0], e3_conv.rules_from_abi(*rules), 6, 400)
        bf = mod.BestFirst(3, 4, 5, rules, 6, k=1)
        levels = bf.run(maps[0], 400)
        if (levels[-1]["visited"], (levels[-1]["best_reward"], levels[-1]["best_visit"]),
                bf_expanded(bf)) != want:
            return False
    root, rules = two_goals()
    levels = mod.BestFirst(3, 3, 4, rules, 100, k=1).run(root, budget=10**6, max_levels=2)
    if (levels[-1]["best_reward"], levels[-1]["best_visit"], levels[-1]["visited"]) != (2, 8, 10):
        return False
    for seed in range(2):
        wl = inputs.Workload("s", 800 + seed, B=1, H=3, W=4, C=5, R=3, shapes=((1, 2), (1, 1)),
                             p_dc=0.6, per_env=False, T=1)
        maps, rules, _ = inputs.make_all(wl, seed, "dense")
        want = textbook_best_first(maps[0], e3_conv.rules_from_abi(*rules), 6, 400)
        bf = mod.BestFirst(3, 4, 5, rules, 6, k=1)
        levels = bf.run(maps[0], 400)
        if (levels[-1]["visited"], (levels[-1]["best_reward"], levels[-1]["best_visit"]),
                bf_expanded(bf)) != want:
            return False
    return True


def test_unmutated_best_first_passes_pins(oracle_lib):
    assert bf_pins(osearch)


@pytest.mark.parametrize("name", sorted(BF_MUTANTS))
def test_best_first_mutant_is_caught(oracle_lib, tmp_path, name):
    old, new = BF_MUTANTS[name]
    src = open(osearch.__file__).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/found"
    path = os.path.join(str(tmp_path), f"bf_{name}.py")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    spec = importlib.util.spec_from_file_location(f"bf_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    assert not bf_pins(mod), f"mutant {name} passes every best-first pin"
