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
        info = dict(parents=len(self.frontier), children=0, terminal=0, survivors=0)
        kids = self._children(self.frontier, max_children)
        if kids:                                        # nothing expanded: frontier kept
            survivors = self._absorb(kids, info)
            self.frontier = [kids[i][:3] for i in survivors[:self.max_frontier]]
            self.level += 1
        info.update(level=self.level, frontier=len(self.frontier), visited=self.visited,
                    best_reward=self.best[0], best_visit=self.best[1])
        return info

    def _absorb(self, kids, info):
        """Count the visits of one expansion's children (in order), track the best node,
        set terminal ones aside and deduplicate the rest against each other and the table.
        Returns the surviving children's indices in increasing order."""
        info["children"] = len(kids)
        best_in_level = {}                             # map -> ((reward, -depth), index)
        for i, (m, reward, depth, done) in enumerate(kids):
            visit = self.visited + 1 + i
            if reward > self.best[0]:
                self.best = (reward, visit)
            if done:
                info["terminal"] += 1
                continue
            key = m.tobytes()
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
        self.visited += len(kids)
        return survivors

    def _children(self, parents, max_children):
        """Step every (parent, action) pair, parents in the given order, cut to max_children.
        parents: list of (map, reward, depth).  Returns [(map, reward, depth, done)]."""
        pairs = [(p, a) for p in range(len(parents)) for a in self.actions][:max(0, max_children)]
        n = len(pairs)
        if n == 0:
            return []
        o = _oracle.Oracle(n, self.H, self.W, self.C, max(self.R, 1), self.mh, self.mw, False,
                           self.L, lib_path=self.lib_path, rule_mode=self.rule_mode)
        o.load_rules(*self.rules)
        o.reset(np.stack([parents[p][0] for p, _ in pairs]))
        o.set_counters(np.array([parents[p][2] for p, _ in pairs], np.int32))
        r, d = o.step(np.array([a for _, a in pairs], np.uint8))
        maps = o.maps()
        o.close()
        return [(maps[i], parents[p][1] + int(r[i]), parents[p][2] + 1, bool(d[i]))
                for i, (p, _) in enumerate(pairs)]

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


class BestFirst(Search):
    """Batched best-first search (the paper scores environments with best-first search that
    prioritises higher reward, Sec. 2.2.1).  Open nodes are ordered by (higher reward, then
    smaller depth, then smaller node id); every iteration pops the k first open nodes (k = 1
    is plain best-first), drops those whose state has since been reached with a better
    (reward, -depth) (the deeper or lower-reward node is pruned), and expands the rest in
    node-id order exactly as one level of Search: children in (parent, action) order cut to
    the remaining budget, terminal children counted and never opened, in-iteration duplicates
    resolved by (reward, -depth) then lowest child index, and a child kept iff its state is new
    or it beats the stored (reward, -depth).  Kept children become open nodes with the next
    ids, in child order.  The root is node 0."""

    def __init__(self, H, W, C, rules, L, k=1, num_actions=5, rule_mode=0,
                 lib_path=_oracle.LIB):
        super().__init__(H, W, C, rules, L, num_actions=num_actions, rule_mode=rule_mode,
                         lib_path=lib_path)
        assert k >= 1
        self.k = k

    def begin(self, root):
        super().begin(root)
        root = self.frontier[0][0]
        self.nodes = [(root, 0, 0)]          # id -> (map, reward, depth)
        self.open = [0]
        self.expanded = []                   # ids of the expanded nodes, in order

    def expand(self, max_children):
        info = dict(parents=0, children=0, terminal=0, survivors=0)
        if max_children <= 0 or not self.open:
            info.update(level=self.level, frontier=len(self.open), visited=self.visited,
                        best_reward=self.best[0], best_visit=self.best[1])
            return info
        self.open.sort(key=lambda i: (-self.nodes[i][1], self.nodes[i][2], i))
        popped, self.open = self.open[:self.k], self.open[self.k:]
        alive = sorted(i for i in popped
                       if self.table[self.nodes[i][0].tobytes()] == (self.nodes[i][1],
                                                                     -self.nodes[i][2]))
        parents = [self.nodes[i] for i in alive]
        self.expanded.extend(alive)
        kids = self._children(parents, max_children)
        info["parents"] = len(parents)
        for i in self._absorb(kids, info):
            m, reward, depth, _ = kids[i]
            self.open.append(len(self.nodes))
            self.nodes.append((m, reward, depth))
        self.level += 1
        info.update(level=self.level, frontier=len(self.open), visited=self.visited,
                    best_reward=self.best[0], best_visit=self.best[1])
        return info

    def open_arrays(self):
        """The open nodes in priority order: (maps, reward, depth, node id)."""
        order = sorted(self.open, key=lambda i: (-self.nodes[i][1], self.nodes[i][2], i))
        if not order:
            return (np.zeros((0, self.C, self.H, self.W), np.uint8), np.zeros(0, np.int32),
                    np.zeros(0, np.int32), np.zeros(0, np.int64))
        return (np.stack([self.nodes[i][0] for i in order]),
                np.array([self.nodes[i][1] for i in order], np.int32),
                np.array([self.nodes[i][2] for i in order], np.int32),
                np.array(order, np.int64))

    def run(self, root, budget, max_levels=1 << 30):
        self.begin(root)
        out = []
        while self.open and self.visited < budget and self.level < max_levels:
            out.append(self.expand(budget - self.visited))
        return out
