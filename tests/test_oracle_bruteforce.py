"""Oracle pinned by exhaustive enumeration on 4x4 maps.

B1  every one of the 2^16 goal planes x every tri-valued 1x2 and 2x1 rule on that channel
    (3^2 input x 3^2 output entries per shape = 162 rules), against the paper's
    convolution form of the step (Sec. 2.1), computed with torch's conv2d /
    conv_transpose2d.
B2  the action phase and built-in moves: every wall plane x every player cell x every
    action, against the closed form "the player moves iff the target cell is on the map
    and holds no wall" (Sec. 2.1 force tiles; Sec. 2.2.1 walls block).
B4  random multi-channel maps, random 2x2 / 3x3 rule sets (force entries included) and
    random actions over several steps, against the convolution form.
"""
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

import e3_conv
import oracle
from paper_2407_04221_amd import inputs

E, W, P, G = 0, 1, 2, 3


def all_planes_4x4():
    k = np.arange(1 << 16, dtype=np.int64)
    bits = (k[:, None] >> np.arange(16)[None, :]) & 1
    return bits.reshape(-1, 4, 4).astype(np.uint8)


def test_b1_single_channel_rules_exhaustive(oracle_lib):
    planes = all_planes_4x4()
    B = planes.shape[0]
    maps = np.zeros((B, 4, 4, 4), np.uint8)
    maps[:, G] = planes
    maps[:, P, 3, 3] = 1          # a player that never moves (no action)
    actions = np.zeros(B, np.uint8)
    xg = torch.from_numpy(planes[:, None].astype(np.float32))
    o = oracle.Oracle(B, 4, 4, 4, 1, 2, 2, False, 0)
    checked = 0
    for n, m in ((1, 2), (2, 1)):
        for ins in itertools.product((-1, 0, 1), repeat=2):
            for outs in itertools.product((-1, 0, 1), repeat=2):
                I = np.full((5, n, m), -1, np.int8)
                O = np.full((5, n, m), -1, np.int8)
                I[G].flat[:] = ins
                O[G].flat[:] = outs
                shape = np.array([[[n, m]]], np.int32)
                ip = np.full((1, 1, 5, 2, 2), -1, np.int8)
                op = np.full((1, 1, 5, 2, 2), -1, np.int8)
                ip[0, 0, :, :n, :m] = I
                op[0, 0, :, :n, :m] = O
                rw = np.array([[1]], np.int32)
                o.load_rules(shape, ip, op, rw)
                o.reset(maps)
                r, d = o.step(actions, nthreads=8)
                got = o.maps()
                # E3 on the goal channel alone: every other kernel entry is zero, and with
                # no action there is no force, so the move rules cannot match
                k_in, thr, k_out = e3_conv.kernels(I[G:G + 1], O[G:G + 1])
                act = torch.relu(Fn.conv2d(xg, k_in.float()) - thr + 1.0)
                new_g = (xg + Fn.conv_transpose2d(act, k_out.float()) >= 1.0)
                want = maps.copy()
                want[:, G] = new_g[:, 0].numpy()
                np.testing.assert_array_equal(got, want, err_msg=f"{n}x{m} in={ins} out={outs}")
                np.testing.assert_array_equal(r, act.sum(dim=(1, 2, 3)).numpy())
                assert not d.any()
                checked += B
    o.close()
    assert checked == 162 * (1 << 16)


def test_b2_moves_exhaustive(oracle_lib):
    walls = all_planes_4x4()
    B = walls.shape[0]
    o = oracle.Oracle(B, 4, 4, 4, 0, 1, 1, False, 0)
    o.load_rules(np.zeros((1, 0, 2), np.int32), np.zeros((1, 0, 5, 1, 1), np.int8),
                 np.zeros((1, 0, 5, 1, 1), np.int8), np.zeros((1, 0), np.int32))
    dirs = {0: (0, 0), 1: (-1, 0), 2: (0, 1), 3: (1, 0), 4: (0, -1)}
    for py in range(4):
        for px in range(4):
            maps = np.zeros((B, 4, 4, 4), np.uint8)
            maps[:, W] = walls
            maps[:, P, py, px] = 1
            for a, (dy, dx) in dirs.items():
                o.reset(maps)
                r, d = o.step(np.full(B, a, np.uint8), nthreads=8)
                got = o.maps()
                ty, tx = py + dy, px + dx
                want = maps.copy()
                if a != 0 and 0 <= ty < 4 and 0 <= tx < 4:
                    free = walls[:, ty, tx] == 0
                    want[free, P, py, px] = 0
                    want[free, P, ty, tx] = 1
                np.testing.assert_array_equal(got, want, err_msg=f"player ({py},{px}) a={a}")
                assert not r.any() and not d.any()
    # action values >= 5 place no force
    maps = np.zeros((B, 4, 4, 4), np.uint8)
    maps[:, W] = walls
    maps[:, P, 1, 1] = 1
    o.reset(maps)
    o.step(np.full(B, 7, np.uint8))
    np.testing.assert_array_equal(o.maps(), maps)
    o.close()


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("variant", ["literal", "planted", "dense"])
def test_b4_random_rule_sets_against_conv_form(oracle_lib, seed, variant):
    # small maps, every channel random (multi-hot), rules over all C+1 channels
    shapes = (((2, 2), (1, 2)), ((3, 3), (2, 1), (1, 1)))[seed % 2]
    wl = inputs.Workload("t", 90 + seed, B=24, H=5 + seed % 3, W=6 + seed % 4, C=4 + seed % 3,
                         R=5, shapes=shapes, p_dc=0.5, per_env=False, T=6, L=4)
    maps, rules, actions = inputs.make_all(wl, seed, variant)
    g = np.random.default_rng(seed)
    noise = (g.random(maps.shape) < 0.25).astype(np.uint8)
    maps = maps | noise      # multi-hot cells, sometimes several players
    want = e3_conv.run(maps, rules, actions, L=wl.L)
    got = oracle.run(wl, maps, rules, actions)
    for k in range(wl.T):
        np.testing.assert_array_equal(got[0][k], want[0][k], err_msg=f"step {k} maps")
        np.testing.assert_array_equal(got[1][k], want[1][k], err_msg=f"step {k} rewards")
        np.testing.assert_array_equal(got[2][k], want[2][k], err_msg=f"step {k} done")


def test_b4_per_env_rule_sets_against_conv_form(oracle_lib):
    wl = inputs.Workload("t", 97, B=6, H=6, W=7, C=5, R=4, shapes=((3, 3), (1, 2), (2, 1)),
                         p_dc=0.6, per_env=True, T=5, L=3)
    maps, rules, actions = inputs.make_all(wl, 3, "planted")
    want = e3_conv.run(maps, rules, actions, L=wl.L, per_env=True)
    got = oracle.run(wl, maps, rules, actions)
    for a, b in zip(got, want):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("variant", ["literal", "planted", "dense"])
def test_b4_sequential_mode_against_conv_form(oracle_lib, seed, variant):
    """Rules applied in sequence: each rule's conv / conv^T pair is applied and clamped
    before the next rule is matched."""
    shapes = (((2, 2), (1, 2)), ((3, 3), (2, 1), (1, 1)))[seed % 2]
    wl = inputs.Workload("t", 110 + seed, B=20, H=5 + seed % 3, W=6 + seed % 4, C=4 + seed % 3,
                         R=5, shapes=shapes, p_dc=0.5, per_env=bool(seed % 2), T=5, L=4)
    maps, rules, actions = inputs.make_all(wl, seed, variant)
    maps = maps | (np.random.default_rng(seed).random(maps.shape) < 0.25).astype(np.uint8)
    want = e3_conv.run(maps, rules, actions, L=wl.L, per_env=wl.per_env, sequential=True)
    got = oracle.run(wl, maps, rules, actions, rule_mode=1)
    for a, b in zip(got, want):
        np.testing.assert_array_equal(a, b)
    par = oracle.run(wl, maps, rules, actions, rule_mode=0)
    if variant != "literal":
        assert not all(np.array_equal(a, b) for a, b in zip(got, par)), \
            "sequential and parallel application should differ on firing rules"
