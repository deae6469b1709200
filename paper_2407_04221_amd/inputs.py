"""Seeded synthetic inputs for the batched rule step: rule sets, initial maps, actions.

This module is the only code shared by the GPU path's callers and by the CPU oracle's
callers.  It draws random numbers and lays them out in the array formats of the C ABI;
it performs none of the step's arithmetic (no matching, voting, clamping or rewards).

Tile roles follow the paper's base maze game (Sec. 2.2.1: player, wall, food/goal, plus
"no-op" tile types that evolution may bring into play): channel 0 = empty, 1 = wall,
2 = player, 3 = goal/food, 4.. = extra tile types.  Channel C (one past the stored ones)
is the transient force plane the player's action creates (Sec. 2.1); rule patterns span
all C+1 channels.

Pattern entries: 1 = must be 1 (in) / becomes 1 (out); 0 = must be 0 / becomes 0;
-1 = don't care (in) / left as is (out).

Random streams: numpy PCG64 seeded by SeedSequence([config_id, seed, stream]) with
stream 0 = rules, 1 = maps, 2 = actions, so each array can be regenerated alone.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Sequence, Tuple

import numpy as np

EMPTY, WALL, PLAYER, GOAL = 0, 1, 2, 3
DONT_CARE = -1

STREAM_RULES, STREAM_MAPS, STREAM_ACTIONS = 0, 1, 2


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: batch shape, rule-set shape and entry distribution."""
    name: str
    config_id: int
    B: int                      # environments
    H: int                      # map rows
    W: int                      # map columns
    C: int                      # stored channels (force plane excluded)
    R: int                      # loaded rules per set
    shapes: Tuple[Tuple[int, int], ...]   # pattern (rows, cols) choices, uniform per rule
    p_dc: float                 # probability that a pattern entry is don't-care
    per_env: bool               # one rule set per environment (else one shared set)
    T: int                      # steps of the workload
    L: int = 100                # episode length (0 = no truncation)
    wall_p: float = 0.3         # probability that an initial cell is a wall

    @property
    def max_h(self) -> int:
        return max(s[0] for s in self.shapes)

    @property
    def max_w(self) -> int:
        return max(s[1] for s in self.shapes)

    @property
    def S(self) -> int:
        return self.B if self.per_env else 1

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads of the benchmark plan: 16x16 single env; 1024 envs with per-env
# rules; 4096 32x32 envs with per-env mixed-shape rules; 16384 envs with one shared set
# (the throughput workload); 256 64x64 envs with 5x5 patterns.
WORKLOADS = {
    "c1": Workload("c1", 1, B=1, H=16, W=16, C=4, R=3, shapes=((3, 3),), p_dc=1.0 / 3.0,
                   per_env=False, T=100),
    "c2": Workload("c2", 2, B=1024, H=16, W=16, C=6, R=8, shapes=((3, 3),), p_dc=0.3,
                   per_env=True, T=1000),
    "c3": Workload("c3", 3, B=4096, H=32, W=32, C=8, R=16,
                   shapes=((3, 3), (1, 2), (2, 1)), p_dc=0.3, per_env=True, T=1000),
    "c4": Workload("c4", 4, B=16384, H=16, W=16, C=6, R=8, shapes=((3, 3),), p_dc=0.3,
                   per_env=False, T=5000),
    "c5": Workload("c5", 5, B=256, H=64, W=64, C=12, R=32, shapes=((5, 5),), p_dc=0.4,
                   per_env=False, T=500),
}

VARIANTS = ("literal", "planted", "dense")


def rng(config_id: int, seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([config_id, seed, stream])))


def make_maps(wl: Workload, seed: int) -> np.ndarray:
    """Initial maps, uint8 [B][C][H][W] in {0,1}.

    Each cell is a wall with probability wl.wall_p, otherwise one tile drawn uniformly
    from {empty, goal, extra types}; then one uniformly chosen cell per map is overwritten
    to hold exactly the player tile.
    """
    g = rng(wl.config_id, seed, STREAM_MAPS)
    B, C, H, W = wl.B, wl.C, wl.H, wl.W
    others = np.array([EMPTY, GOAL] + list(range(4, C)), dtype=np.int64)
    is_wall = g.random((B, H, W)) < wl.wall_p
    pick = others[g.integers(0, len(others), size=(B, H, W))]
    tile = np.where(is_wall, WALL, pick)
    pos = g.integers(0, H * W, size=B)
    tile = tile.reshape(B, H * W)
    tile[np.arange(B), pos] = PLAYER
    tile = tile.reshape(B, H, W)
    maps = np.zeros((B, C, H, W), dtype=np.uint8)
    for c in range(C):
        maps[:, c] = (tile == c)
    return maps


def _draw_entries(g: np.random.Generator, size, p_dc: float) -> np.ndarray:
    dc = g.random(size) < p_dc
    bit = g.integers(0, 2, size=size)
    return np.where(dc, DONT_CARE, bit).astype(np.int8)


def make_rules(wl: Workload, seed: int, variant: str = "literal",
               init_maps: Optional[np.ndarray] = None):
    """Rule sets in the ABI's layout.

    Returns (shape int32 [S][R][2], in_pat int8 [S][R][C+1][mh][mw],
    out_pat int8 [S][R][C+1][mh][mw], reward int32 [S][R]); entries outside a rule's own
    rows x cols are don't-care.

    variant:
      literal  entries i.i.d.: don't-care with prob p_dc, else 0/1 with prob 1/2 each;
      dense    the same with input p_dc = 0.9 (rules fire on most of the map);
      planted  as literal, then every specified input entry of the stored channels is
               overwritten with the value found at one random valid position of the
               set's initial map (env 0's map for a shared set), and force-plane input
               entries become don't-care, so each rule matches at least once at t = 0.
    """
    if variant not in VARIANTS:
        raise ValueError(f"unknown variant {variant!r}")
    g = rng(wl.config_id, seed, STREAM_RULES)
    S, R, C1, mh, mw = wl.S, wl.R, wl.C + 1, wl.max_h, wl.max_w
    shape_idx = g.integers(0, len(wl.shapes), size=(S, R))
    shape = np.array(wl.shapes, dtype=np.int32)[shape_idx].reshape(S, R, 2)
    p_in = 0.9 if variant == "dense" else wl.p_dc
    in_pat = _draw_entries(g, (S, R, C1, mh, mw), p_in)
    out_pat = _draw_entries(g, (S, R, C1, mh, mw), wl.p_dc)
    reward = g.integers(-1, 2, size=(S, R)).astype(np.int32)
    # entries outside each rule's own rows x cols are don't-care
    rows = np.arange(mh)[None, None, None, :, None]
    cols = np.arange(mw)[None, None, None, None, :]
    inside = (rows < shape[:, :, 0][:, :, None, None, None]) & \
             (cols < shape[:, :, 1][:, :, None, None, None])
    in_pat = np.where(inside, in_pat, DONT_CARE).astype(np.int8)
    out_pat = np.where(inside, out_pat, DONT_CARE).astype(np.int8)
    if variant == "planted":
        if init_maps is None:
            raise ValueError("planted rules need the initial maps")
        for s in range(S):
            m = init_maps[s]
            for r in range(R):
                n_, m_ = int(shape[s, r, 0]), int(shape[s, r, 1])
                ay = int(g.integers(0, wl.H - n_ + 1))
                ax = int(g.integers(0, wl.W - m_ + 1))
                patch = m[:, ay:ay + n_, ax:ax + m_].astype(np.int8)
                blk = in_pat[s, r, :wl.C, :n_, :m_]
                in_pat[s, r, :wl.C, :n_, :m_] = np.where(blk == DONT_CARE, DONT_CARE, patch)
                in_pat[s, r, wl.C] = DONT_CARE
    return shape, in_pat, out_pat, reward


def make_actions(wl: Workload, seed: int, T: Optional[int] = None) -> np.ndarray:
    """Actions uint8 [T][B], i.i.d. uniform over {0: none, 1: up, 2: right, 3: down, 4: left}."""
    g = rng(wl.config_id, seed, STREAM_ACTIONS)
    T = wl.T if T is None else T
    return g.integers(0, 5, size=(T, wl.B)).astype(np.uint8)


def make_all(wl: Workload, seed: int, variant: str = "literal", T: Optional[int] = None):
    """(maps, (shape, in_pat, out_pat, reward), actions) for one workload and seed."""
    maps = make_maps(wl, seed)
    rules = make_rules(wl, seed, variant, init_maps=maps)
    actions = make_actions(wl, seed, T)
    return maps, rules, actions


def subset_envs(wl: Workload, maps: np.ndarray, rules, actions: np.ndarray,
                envs: Sequence[int]):
    """Restrict a workload's arrays to some environments (envs are independent)."""
    envs = np.asarray(envs, dtype=np.int64)
    shape, in_pat, out_pat, reward = rules
    if wl.per_env:
        rules = (shape[envs], in_pat[envs], out_pat[envs], reward[envs])
    return maps[envs], rules, actions[:, envs]
