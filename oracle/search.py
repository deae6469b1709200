"""Level-synchronous search over action sequences with state deduplication, on the CPU.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only the tests and the benchmark's CPU
baseline use it; it steps states with the oracle (oracle/avo.c) and shares nothing with
the GPU library.

The paper scores an environment by searching the action sequences a player can take and
counting the states visited before the highest-reward solution is found (Sec. 2.2.1).  A
node is a game state: the map (which holds the player's position), the reward accumulated
on the way, and its depth; an edge is an action.  A state equal to one seen before keeps
the node with the higher reward, and among equal rewards the shallower one; the other is
pruned.  This search expands whole levels (breadth-first, the budgeted search the paper
also names), which makes every level one batched step of all parent x action pairs:

  level d: children = (parent, action) for every node of the frontier in order, then every
           action in order, cut to the remaining budget of visits;
           each child is the parent's map stepped once with the action (the step counter
           starts at the parent's depth, so a child at depth L ends its episode);
           visit index of child i = visits so far + 1 + i (the root is visit 0);
           reward = parent reward + step reward; the best (highest reward, earliest visit)
           is tracked over the root and every child;
           children whose episode ended are terminal (counted, never expanded);
           the others are grouped by map: the best of a group by (reward, -depth), lowest
           index among equals, survives iff its map is new or it beats the stored
           (reward, -depth) of that map; survivors, in index order, cut to max_frontier,
           are the next frontier.
"""
from __future__ import annotations

import numpy as np

import oracle as _oracle


class Search:
    def __init__(self, H, W, C, rules, L, num_actions=5, max_frontier=1 << 20, rule_mode=0,
                 lib_path=_oracle.LIB):
        shape, ip, op, rw = rules
        assert shape.shape[0] == 1, "one rule set"
        assert num_actions in (4, 5)
        self.H, self.W, self.C, self.L = H, W, C, L
        self.rules = (shape, ip, op, rw)
        self.R, self.mh, self.mw = shape.shape[1], ip.shape[3], ip.shape[4]
        self.actions = list(range(5)) if num_actions == 5 else [1, 2, 3, 4]
        self.max_frontier = max_frontier
        self.rule_mode = rule_mode
        self.lib_path = lib_path

    def begin(self, root):
        root = (np.asarray(root) != 0).astype(np.uint8)
        self.frontier = [(root, 0, 0)]                 # (map, reward, depth)
        self.table = {root.tobytes(): (0, 0)}          # map -> (reward, -depth), best kept
        self.visited = 0
        self.level = 0
        self.best = (0, 0)                             # (reward, visit index)

    def expand(self, max_children):
        A = len(self.actions)
        pairs = [(p, a) for p in range(len(self.frontier)) for a in self.actions]
        pairs = pairs[:max(0, max_children)]
        n = len(pairs)
        info = dict(parents=len(self.frontier), children=n, terminal=0, survivors=0)
        if n == 0:                                      # nothing expanded: frontier kept
            info.update(level=self.level, frontier=0, visited=self.visited,
                        best_reward=self.best[0], best_visit=self.best[1])
            return info
        o = _oracle.Oracle(n, self.H, self.W, self.C, max(self.R, 1), self.mh, self.mw, False,
                           self.L, lib_path=self.lib_path, rule_mode=self.rule_mode)
        o.load_rules(*self.rules)
        o.reset(np.stack([self.frontier[p][0] for p, _ in pairs]))
        o.set_counters(np.array([self.frontier[p][2] for p, _ in pairs], np.int32))
        r, d = o.step(np.array([a for _, a in pairs], np.uint8))
        maps = o.maps()
        o.close()
        best_in_level = {}                             # map -> ((reward, -depth), index)
        kids = []
        for i, (p, a) in enumerate(pairs):
            reward = self.frontier[p][1] + int(r[i])
            depth = self.frontier[p][2] + 1
            visit = self.visited + 1 + i
            if reward > self.best[0]:
                self.best = (reward, visit)
            kids.append((maps[i], reward, depth))
            if d[i]:
                info["terminal"] += 1
                continue
            key = maps[i].tobytes()
            val = (reward, -depth)
            if key not in best_in_level or val > best_in_level[key][0]:
                best_in_level[key] = (val, i)
        survivors = []
        for key, (val, i) in best_in_level.items():
            old = self.table.get(key)
            if old is None or val > old:
                self.table[key] = val
                survivors.append(i)
        survivors.sort()
        info["survivors"] = len(survivors)
        self.frontier = [kids[i] for i in survivors[:self.max_frontier]]
        self.visited += n
        self.level += 1
        info.update(level=self.level, frontier=len(self.frontier), visited=self.visited,
                    best_reward=self.best[0], best_visit=self.best[1])
        return info

    def frontier_arrays(self):
        """(maps uint8 [N][C][H][W], reward int32 [N], depth int32 [N]) in frontier order."""
        if not self.frontier:
            return (np.zeros((0, self.C, self.H, self.W), np.uint8), np.zeros(0, np.int32),
                    np.zeros(0, np.int32))
        return (np.stack([f[0] for f in self.frontier]),
                np.array([f[1] for f in self.frontier], np.int32),
                np.array([f[2] for f in self.frontier], np.int32))

    def run(self, root, budget, max_levels=1 << 30):
        """Expand levels until the frontier is empty, the budget of visits is spent or
        max_levels is reached; returns the list of per-level infos."""
        self.begin(root)
        out = []
        while self.frontier and self.visited < budget and self.level < max_levels:
            out.append(self.expand(budget - self.visited))
        return out
