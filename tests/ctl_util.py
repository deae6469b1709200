"""Seeded rule application control for tests: per-rule limits and inhibition masks."""
import numpy as np


def random_control(g, S, R, p_limit=0.6, p_inh=0.3, kmax=3):
    """limit int32 [S][R] (0 or 1..kmax), inhibit uint8 [S][R][R] with q < r only."""
    limit = np.where(g.random((S, R)) < p_limit, g.integers(1, kmax + 1, (S, R)), 0)
    inhibit = (g.random((S, R, R)) < p_inh).astype(np.uint8)
    inhibit *= np.triu(np.ones((R, R), np.uint8), 1)[None]
    return limit.astype(np.int32), inhibit
