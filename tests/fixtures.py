"""Parser for the hand-worked step fixtures in tests/golden/*.av.

Format (line based, '#' starts a comment):

    mode sequential              optional: rules applied one after another (default parallel)
    channels <C>                 stored channels; tiles E W P G a b c ... (0, 1, 2, 3, 4 ...)
    episode <L>                  optional episode length (default 0 = none)
    order rowmajor|random        optional rule application control (site order, default
    seed <s>                     row-major) and the key of the random index channel
    rule <n>x<m> reward <r>      one block per loaded rule, in index order
    in  <i>,<j> <T>=<v> ... | <i>,<j> <T>=<v> ...     specified input entries
    out <i>,<j> <T>=<v> ... | ...                     specified output entries
    limit <K>                    optional: at most K matches of this rule apply per step
    inhibits <q>                 optional: this rule is inhibited by earlier rule q
    map                          the initial map follows, one line per row
    step <action>                one block per step: the map after the step follows,
    reward <r>                   then the step's reward
    done <d>                     and done flag

Map cells are '.' (no tile) or the letters of the tiles present, e.g. 'PG'.  In rule
entries T may also be F (the force plane, channel C).  Unlisted entries are don't care.
"""
from __future__ import annotations

import os
from dataclasses import dataclass, field
from typing import List

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TILES = "EWPG" + "abcdefghijklmnopqrstuvwxyz"


def tile_index(ch: str, C: int) -> int:
    if ch == "F":
        return C
    k = TILES.index(ch)
    if k >= C:
        raise ValueError(f"tile {ch!r} needs more than {C} channels")
    return k


@dataclass
class Step:
    action: int
    after: np.ndarray
    reward: float
    done: int


@dataclass
class Fixture:
    name: str
    C: int
    L: int
    mode: int = 0                                # 0 parallel, 1 sequential
    order: int = 0                               # 0 row-major, 1 random index channel
    seed: int = 0
    limits: dict = field(default_factory=dict)   # rule -> K
    inhibits: list = field(default_factory=list)  # (q, r): q inhibits r
    rules: list = field(default_factory=list)   # (n, m, in [C+1][n][m], out, reward)
    init: np.ndarray = None                      # [C][H][W]
    steps: List[Step] = field(default_factory=list)

    @property
    def H(self):
        return self.init.shape[1]

    @property
    def W(self):
        return self.init.shape[2]

    def abi_rules(self):
        """Rules as ABI arrays for one shared set (S = 1)."""
        R = len(self.rules)
        mh = max([r[0] for r in self.rules] + [1])
        mw = max([r[1] for r in self.rules] + [1])
        shape = np.zeros((1, R, 2), np.int32)
        ip = np.full((1, R, self.C + 1, mh, mw), -1, np.int8)
        op = np.full((1, R, self.C + 1, mh, mw), -1, np.int8)
        rw = np.zeros((1, R), np.int32)
        for k, (n, m, i_, o_, r_) in enumerate(self.rules):
            shape[0, k] = (n, m)
            ip[0, k, :, :n, :m] = i_
            op[0, k, :, :n, :m] = o_
            rw[0, k] = r_
        return shape, ip, op, rw, mh, mw


    @property
    def has_control(self):
        return bool(self.limits or self.inhibits or self.order)

    def abi_control(self):
        """(limit [1][R], inhibit [1][R][R], order, seed) for one shared set."""
        R = len(self.rules)
        limit = np.zeros((1, R), np.int32)
        inhibit = np.zeros((1, R, R), np.uint8)
        for r, k in self.limits.items():
            limit[0, r] = k
        for q, r in self.inhibits:
            inhibit[0, q, r] = 1
        return limit, inhibit, self.order, self.seed


def _parse_cells(line: str, C: int, W: int = None) -> np.ndarray:
    toks = line.split()
    row = np.zeros((C, len(toks)), np.uint8)
    for x, t in enumerate(toks):
        if t == ".":
            continue
        for ch in t:
            row[tile_index(ch, C), x] = 1
    return row


def _parse_entries(text: str, C: int, n: int, m: int) -> np.ndarray:
    pat = np.full((C + 1, n, m), -1, np.int8)
    for group in text.split("|"):
        group = group.strip()
        if not group:
            continue
        pos, *assigns = group.split()
        i, j = (int(v) for v in pos.split(","))
        for a in assigns:
            t, v = a.split("=")
            pat[tile_index(t, C), i, j] = int(v)
    return pat


def parse(path: str) -> Fixture:
    name = os.path.splitext(os.path.basename(path))[0]
    lines = []
    with open(path) as f:
        for raw in f:
            s = raw.split("#", 1)[0].rstrip()
            if s.strip():
                lines.append(s.strip())
    fx = Fixture(name=name, C=0, L=0)
    k = 0
    keywords = ("mode", "channels", "episode", "rule", "in", "out", "map", "step", "reward",
                "done", "limit", "inhibits", "order", "seed")

    def grab_rows(k):
        rows = []
        while k < len(lines) and lines[k].split()[0] not in keywords:
            rows.append(_parse_cells(lines[k], fx.C))
            k += 1
        return np.stack(rows, axis=1), k   # [C][H][W]

    while k < len(lines):
        head, *rest = lines[k].split(None, 1)
        rest = rest[0] if rest else ""
        k += 1
        if head == "mode":
            fx.mode = {"parallel": 0, "sequential": 1}[rest.strip()]
        elif head == "order":
            fx.order = {"rowmajor": 0, "random": 1}[rest.strip()]
        elif head == "seed":
            fx.seed = int(rest)
        elif head == "limit":
            fx.limits[len(fx.rules) - 1] = int(rest)
        elif head == "inhibits":
            fx.inhibits.append((int(rest), len(fx.rules) - 1))
        elif head == "channels":
            fx.C = int(rest)
        elif head == "episode":
            fx.L = int(rest)
        elif head == "rule":
            size, _, r = rest.split()
            n, m = (int(v) for v in size.split("x"))
            fx.rules.append([n, m, np.full((fx.C + 1, n, m), -1, np.int8),
                             np.full((fx.C + 1, n, m), -1, np.int8), int(r)])
        elif head == "in":
            n, m = fx.rules[-1][0], fx.rules[-1][1]
            fx.rules[-1][2] = _parse_entries(rest, fx.C, n, m)
        elif head == "out":
            n, m = fx.rules[-1][0], fx.rules[-1][1]
            fx.rules[-1][3] = _parse_entries(rest, fx.C, n, m)
        elif head == "map":
            fx.init, k = grab_rows(k)
        elif head == "step":
            after, k = grab_rows(k)
            fx.steps.append(Step(int(rest), after, 0.0, 0))
        elif head == "reward":
            fx.steps[-1].reward = float(rest)
        elif head == "done":
            fx.steps[-1].done = int(rest)
        else:
            raise ValueError(f"{path}: unknown keyword {head!r}")
    fx.rules = [tuple(r) for r in fx.rules]
    return fx


def all_fixtures():
    return sorted(os.path.join(GOLDEN, f) for f in os.listdir(GOLDEN) if f.endswith(".av"))
