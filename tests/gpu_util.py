"""Helpers for the GPU tests: run the HIP path through the C ABI on the same seeded
arrays the oracle gets."""
import sys

import numpy as np
import pytest

import paper_2407_04221_amd as av


def rows_ok(wl):
    """The rows engine takes at most 64 rules with the moves and, within 64 KiB of LDS,
    C + 2 planes, 2 (C + 1) vote planes and one match plane per rule (H + 16 rows each, the
    match planes 16 more; 4 bytes per row for W <= 32, else 8) plus 36 bytes per rule and 96
    for the helper waves' candidate masks and shared counters."""
    rt = wl.R + 4
    rowb = 4 if wl.W <= 32 else 8
    hp = wl.H + 16
    lds = ((wl.C + 2 + 2 * (wl.C + 1)) * hp + rt * (hp + 16)) * rowb + 36 * rt + 96
    return rt <= 64 and lds <= 65536


def group_ok(wl, rule_mode="parallel"):
    """The group engine takes maps of at most 32 x 32 in parallel rule order with (R + 4) x
    pattern cells <= 254, at most 8 channels per lane group and 16 rules per group (4 groups of
    16 lanes, covering 16 rows, or 32 with two rows a lane), and within 64 KiB of LDS: C + 1
    planes and R + 4 match planes of PR = HR + ph - 1 rows (rounded up to 4), 3 C rows of HR
    (votes, initial rows), a 12-word probe row per rule plus one, and a word per channel and rule
    plus two; the stored and force planes' rows addressed in 12 bits."""
    if rule_mode != "parallel" or wl.H > 32 or wl.W > 32:
        return False
    rt = wl.R + 4
    hr = 16 if wl.H <= 16 else 32
    G = 4
    pr = (hr + wl.max_h - 1 + 3) & ~3
    lds = 4 * ((wl.C + 1) * pr + rt * pr + 3 * wl.C * hr + (rt + 1) * 12 + wl.C * (rt + 2))
    return (rt * wl.max_h * wl.max_w <= 254 and rt <= 16 * G and rt <= 64 and wl.C <= 8 * G
            and (wl.C + 1) * pr <= 4096 and lds <= 65536)


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    av.load_library()          # missing library = failure, not a skip


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def gpu_run(wl, maps, rules, actions, engine="auto", mode="step", chunk=7, B=None,
            per_step_maps=True, rule_mode="parallel", control=None):
    """Returns (maps per step or None, final maps, rewards [T][B], done [T][B]) as numpy,
    and the engine the batch used.  control: None or (limit, inhibit, order, seed)."""
    import torch
    B = maps.shape[0] if B is None else B
    b = av.Batch.for_workload(wl, B=B, engine=engine, rule_mode=rule_mode)
    try:
        b.load_rules(*rules)
        if control is not None:
            b.set_rule_control(*control)
        b.reset(maps)
        T = actions.shape[0]
        acts = torch.from_numpy(np.ascontiguousarray(actions)).cuda()
        seq = [] if (mode == "step" and per_step_maps) else None
        if mode == "step":
            rs, ds = [], []
            for t in range(T):
                r, d = b.step(acts[t])
                rs.append(r.clone())
                ds.append(d.clone())
                if seq is not None:
                    seq.append(b.maps().cpu().numpy())
            rewards = torch.stack(rs).cpu().numpy()
            done = torch.stack(ds).cpu().numpy()
        else:
            rewards = torch.empty((T, B), dtype=torch.float32, device="cuda")
            done = torch.empty((T, B), dtype=torch.uint8, device="cuda")
            for t0 in range(0, T, chunk):
                k = min(chunk, T - t0)
                b.step_n(acts[t0:t0 + k], rewards[t0:t0 + k], done[t0:t0 + k])
            rewards = rewards.cpu().numpy()
            done = done.cpu().numpy()
        final = b.maps().cpu().numpy()
        torch.cuda.synchronize()
        eng = b.info["engine"]
    finally:
        b.close()
    return (None if seq is None else np.stack(seq)), final, rewards, done, eng


def first_mismatch(a, b):
    idx = np.argwhere(a != b)
    return tuple(idx[0]) if len(idx) else None
