"""Batched search on the GPU (av_search_*) vs the oracle's level-synchronous search
(oracle/search.py): every level's counts, best reward and visit, and the whole frontier
(maps, rewards, depths, in order) compared exactly, for every workload's map shape and rule
set, both action sets, episode ends, frontier and budget cuts, both rule orders and every
step engine; plus a table that overflows (an error, not a fault)."""
import numpy as np
import pytest

from gpu_util import require_gpu, say
import paper_2407_04221_amd as av
from paper_2407_04221_amd import inputs
from oracle import search as osearch

pytestmark = pytest.mark.gpu


def one_set(rules):
    shape, ip, op, rw = rules
    return shape[:1], ip[:1], op[:1], rw[:1]


def compare(wl, root, rules, budget, levels, A=5, cap=1 << 12, L=None, engine="auto",
            rule_mode="parallel", table_log2=18, hash_bits=0):
    L = wl.L if L is None else L
    mode = int(rule_mode == "sequential")
    o = osearch.Search(wl.H, wl.W, wl.C, rules, L, num_actions=A, max_frontier=cap,
                       rule_mode=mode)
    g = av.Search(wl.H, wl.W, wl.C, wl.R, wl.max_h, wl.max_w, L, num_actions=A,
                  max_frontier=cap, table_log2=table_log2, engine=engine, rule_mode=rule_mode,
                  hash_bits=hash_bits)
    try:
        g.load_rules(*rules)
        o.begin(root)
        g.begin(root)
        for lv in range(levels):
            left = budget - o.visited
            want = o.expand(left)
            got = g.expand(left)
            assert got == want, f"level {lv + 1}: {got} != {want}"
            gm, gr, gd = (x.cpu().numpy() for x in g.frontier())
            om, orw, od = o.frontier_arrays()
            np.testing.assert_array_equal(gm, om, err_msg=f"level {lv + 1} maps")
            np.testing.assert_array_equal(gr, orw, err_msg=f"level {lv + 1} rewards")
            np.testing.assert_array_equal(gd, od, err_msg=f"level {lv + 1} depths")
            if want["frontier"] == 0 or want["visited"] >= budget:
                break
        return want
    finally:
        g.close()


CASES = [("c1", 4000, 12), ("c2", 3000, 10), ("c3", 2000, 6), ("c4", 4000, 12), ("c5", 600, 4)]


@pytest.mark.parametrize("variant", ["planted", "dense"])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_search_matches_oracle(case, variant):
    require_gpu()
    name, budget, levels = case
    wl = inputs.WORKLOADS[name].with_(B=1)
    say(f"[search] {name} {variant}")
    maps, rules, _ = inputs.make_all(wl, 7, variant)
    last = compare(wl, maps[0], one_set(rules), budget, levels)
    assert last["visited"] > 0


@pytest.mark.parametrize("engine", ["generic", "wave", "lane16", "rows"])
def test_search_engines_and_options(engine):
    require_gpu()
    wl = inputs.WORKLOADS["c4"].with_(B=1)
    say(f"[search options] engine={engine}")
    maps, rules, _ = inputs.make_all(wl, 3, "planted")
    rules = one_set(rules)
    compare(wl, maps[0], rules, 3000, 10, engine=engine)
    compare(wl, maps[0], rules, 3000, 10, A=4, engine=engine)
    compare(wl, maps[0], rules, 2500, 8, cap=37, engine=engine)          # frontier cut
    compare(wl, maps[0], rules, 777, 8, engine=engine)                    # budget cut mid-level
    compare(wl, maps[0], rules, 3000, 8, L=3, engine=engine)              # level-3 terminal
    compare(wl, maps[0], rules, 3000, 8, engine=engine, rule_mode="sequential")


def test_search_odd_shapes():
    require_gpu()
    for H, W, C in ((5, 7, 5), (33, 9, 4), (2, 64, 6)):
        wl = inputs.Workload("odd", 90 + H, B=1, H=H, W=W, C=C, R=4,
                             shapes=((1, 2), (2, 1), (2, 2)), p_dc=0.5, per_env=False, T=1, L=9)
        say(f"[search odd] {H}x{W} C={C}")
        maps, rules, _ = inputs.make_all(wl, 1, "dense")
        compare(wl, maps[0], rules, 1500, 8)


@pytest.mark.parametrize("hash_bits", [1, 3, 10])
@pytest.mark.parametrize("name", ["c4", "c3"])
def test_search_states_compared_exactly(name, hash_bits):
    """With only the low 1, 3 or 10 bits of the map hash kept, most distinct states share a
    hash with others (paper Sec. 2.2.1 prunes equal states only): the levels must still equal
    the oracle's, which compares maps exactly."""
    require_gpu()
    wl = inputs.WORKLOADS[name].with_(B=1)
    say(f"[search exact] {name} hash_bits={hash_bits}")
    maps, rules, _ = inputs.make_all(wl, 5, "dense")
    budget = 2500 if name == "c4" else 1200
    last = compare(wl, maps[0], one_set(rules), budget, 10, hash_bits=hash_bits)
    assert last["visited"] > 0 and last["survivors"] > 1


def test_search_table_overflow_is_an_error():
    require_gpu()
    wl = inputs.WORKLOADS["c1"].with_(B=1)
    maps, rules, _ = inputs.make_all(wl, 0, "planted")
    g = av.Search(wl.H, wl.W, wl.C, wl.R, wl.max_h, wl.max_w, 100, max_frontier=4096,
                  table_log2=4)
    try:
        g.load_rules(*rules)
        g.begin(maps[0])
        with pytest.raises(av.AvError) as e:
            for _ in range(20):
                g.expand(10**6)
        assert e.value.status == av.AV_ENOMEM
        g.begin(maps[0])                          # a fresh start works again
        assert g.expand(5)["children"] == 5
    finally:
        g.close()


def compare_best_first(wl, root, rules, budget, iters, k, A=5, L=None, engine="auto",
                       rule_mode="parallel", max_nodes=1 << 16, table_log2=18, hash_bits=0):
    L = wl.L if L is None else L
    mode = int(rule_mode == "sequential")
    o = osearch.BestFirst(wl.H, wl.W, wl.C, rules, L, k=k, num_actions=A, rule_mode=mode)
    g = av.Search(wl.H, wl.W, wl.C, wl.R, wl.max_h, wl.max_w, L, num_actions=A,
                  table_log2=table_log2, engine=engine, rule_mode=rule_mode, best_first_k=k,
                  max_nodes=max_nodes, hash_bits=hash_bits)
    try:
        g.load_rules(*rules)
        o.begin(root)
        g.begin(root)
        want = None
        for it in range(iters):
            left = budget - o.visited
            want = o.expand(left)
            got = g.expand(left)
            assert got == want, f"iteration {it + 1}: {got} != {want}"
            gm, gr, gd = (x.cpu().numpy() for x in g.frontier())
            om, orw, od, _ = o.open_arrays()
            np.testing.assert_array_equal(gr, orw, err_msg=f"iteration {it + 1} rewards")
            np.testing.assert_array_equal(gd, od, err_msg=f"iteration {it + 1} depths")
            np.testing.assert_array_equal(gm, om, err_msg=f"iteration {it + 1} maps")
            if want["frontier"] == 0 or want["visited"] >= budget:
                break
        return want
    finally:
        g.close()


BF_CASES = [("c1", 3000, 30), ("c2", 2000, 25), ("c3", 1500, 12), ("c4", 3000, 30), ("c5", 400, 6)]


@pytest.mark.parametrize("k", [1, 7, 64, 512])
@pytest.mark.parametrize("variant", ["planted", "dense"])
@pytest.mark.parametrize("case", BF_CASES, ids=[c[0] for c in BF_CASES])
def test_best_first_matches_oracle(case, variant, k):
    require_gpu()
    name, budget, iters = case
    wl = inputs.WORKLOADS[name].with_(B=1)
    say(f"[best-first] {name} {variant} k={k}")
    maps, rules, _ = inputs.make_all(wl, 5, variant)
    last = compare_best_first(wl, maps[0], one_set(rules), budget, iters, k)
    assert last["visited"] > 0


@pytest.mark.parametrize("engine", ["generic", "wave", "lane16", "rows"])
def test_best_first_engines_and_options(engine):
    require_gpu()
    wl = inputs.WORKLOADS["c4"].with_(B=1)
    say(f"[best-first options] engine={engine}")
    maps, rules, _ = inputs.make_all(wl, 3, "planted")
    rules = one_set(rules)
    compare_best_first(wl, maps[0], rules, 2000, 20, 16, engine=engine)
    compare_best_first(wl, maps[0], rules, 2000, 20, 16, A=4, engine=engine)
    compare_best_first(wl, maps[0], rules, 333, 20, 64, engine=engine)          # budget cut
    compare_best_first(wl, maps[0], rules, 2000, 20, 8, L=3, engine=engine)     # terminal
    compare_best_first(wl, maps[0], rules, 2000, 12, 8, engine=engine, rule_mode="sequential")


@pytest.mark.parametrize("hash_bits", [2, 12])
def test_best_first_states_compared_exactly(hash_bits):
    """Best-first with most states sharing a truncated map hash: the iterations, including
    the liveness test of popped nodes against their state's slot, equal the oracle's."""
    require_gpu()
    wl = inputs.WORKLOADS["c4"].with_(B=1)
    say(f"[best-first exact] hash_bits={hash_bits}")
    maps, rules, _ = inputs.make_all(wl, 5, "dense")
    last = compare_best_first(wl, maps[0], one_set(rules), 2000, 25, 16, hash_bits=hash_bits)
    assert last["visited"] > 0


def test_best_first_pool_full_is_an_error():
    require_gpu()
    wl = inputs.WORKLOADS["c1"].with_(B=1)
    maps, rules, _ = inputs.make_all(wl, 0, "planted")
    g = av.Search(wl.H, wl.W, wl.C, wl.R, wl.max_h, wl.max_w, 100, best_first_k=32,
                  max_nodes=40)
    try:
        g.load_rules(*rules)
        g.begin(maps[0])
        with pytest.raises(av.AvError) as e:
            for _ in range(50):
                g.expand(10**6)
        assert e.value.status == av.AV_ENOMEM
        g.begin(maps[0])
        assert g.expand(5)["children"] == 5
    finally:
        g.close()


def test_best_first_force_pays_skips_dominated_nodes():
    """A rule that pays for every force tile re-reaches states with more reward all the time;
    the earlier open copies are popped and skipped (iterations with no parent)."""
    require_gpu()
    import test_oracle_search as tos
    root, rules = tos.force_pays()
    wl = inputs.Workload("fp", 1, B=1, H=1, W=3, C=4, R=1, shapes=((1, 1),), p_dc=0.0,
                         per_env=False, T=1, L=5)
    last = compare_best_first(wl, root, rules, 200, 100, 1, L=5)
    assert last["frontier"] == 0
