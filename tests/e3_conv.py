"""The step written as the paper's convolution pair (Sec. 2.1), with torch CPU library
convolutions in float64.  Used only as an independent pin of the oracle: the oracle
loops over anchors and entries; this module never does.

    B_t     = ReLU(conv_{K_I}(D_t) - I + 1)          (match activation)
    D_{t+1} = conv^T_{K_O}(B_t) + D_t                 (write), then clamped to {0, 1}

K_I holds +1 for a must-be-1 entry, -1 for must-be-0 and 0 for don't care; I is the
number of +1 entries.  K_O = O - I, with don't-cares resolved so that an unspecified
output leaves the cell alone and an unspecified input points the vote at the output.
No padding: patterns lie wholly on the map.
"""
from __future__ import annotations

import numpy as np
import torch
import torch.nn.functional as Fn

PLAYER, WALL = 2, 1


def move_rules(C: int):
    """Built-in moves as (n, m, I, O, reward); force plane is channel C.
    Moving right: player at (0,0), force on a wall-free cell at (0,1)."""
    out = []
    # (n, m, source cell, target cell)
    for n, m, src, tgt in ((1, 2, (0, 0), (0, 1)), (1, 2, (0, 1), (0, 0)),
                           (2, 1, (0, 0), (1, 0)), (2, 1, (1, 0), (0, 0))):
        I = np.full((C + 1, n, m), -1, np.int8)
        O = np.full((C + 1, n, m), -1, np.int8)
        I[(PLAYER,) + src] = 1
        O[(PLAYER,) + src] = 0
        I[(C,) + tgt] = 1
        I[(WALL,) + tgt] = 0
        O[(PLAYER,) + tgt] = 1
        O[(C,) + tgt] = 0
        out.append((n, m, I, O, 0))
    return out


def kernels(I: np.ndarray, O: np.ndarray):
    I = I.astype(np.int64)
    O = O.astype(np.int64)
    k_in = np.where(I == 1, 1.0, np.where(I == 0, -1.0, 0.0))
    thr = float((I == 1).sum())
    i_eff = np.where(I == -1, 1 - O, I)         # unspecified input: opposite of the output
    o_eff = np.where(O == -1, i_eff, O)         # unspecified output: equal to the input
    k_out = (o_eff - i_eff).astype(np.float64)
    return (torch.from_numpy(k_in)[None].double(), thr,
            torch.from_numpy(k_out)[None].double())


def force_plane(P: torch.Tensor, actions: np.ndarray) -> torch.Tensor:
    """P: [B][H][W]; force on the on-map neighbour of every player cell in the action's
    direction (1 up, 2 right, 3 down, 4 left)."""
    F = torch.zeros_like(P)
    a = torch.from_numpy(np.asarray(actions, dtype=np.int64))
    up, right, down, left = (a == 1), (a == 2), (a == 3), (a == 4)
    F[up, :-1, :] = P[up, 1:, :]
    F[down, 1:, :] = P[down, :-1, :]
    F[right, :, 1:] = P[right, :, :-1]
    F[left, :, :-1] = P[left, :, 1:]
    return F


def site_keys(order: int, seed: int, n: int, b: int, H: int, W: int) -> np.ndarray:
    """Index channel of env b at batch step n over all H*W anchor cells, row-major.
    Row-major order: 4095 - pos.  Random order: numpy's Philox4x64-10 generator with key
    (seed, 0), 32-bit word pos % 8 of the block for counter (pos // 8, n, b, 0) in the high
    20 bits (numpy advances the counter before each block, hence the counter - 1)."""
    pos = np.arange(H * W, dtype=np.int64)
    rank = (4095 - pos).astype(np.uint64)
    if order == 0:
        return rank
    out = np.zeros(H * W, np.uint64)
    for g in range((H * W + 7) // 8):
        ctr = g + (n << 64) + (b << 128)
        bg = np.random.Philox(key=seed, counter=(ctr - 1) % (1 << 256))
        words = bg.random_raw(4)
        for j in range(8):
            p = 8 * g + j
            if p < H * W:
                u = (int(words[j // 2]) >> (32 * (j % 2))) & 0xFFFFFFFF
                out[p] = (u & 0xFFFFF000) | int(rank[p])
    return out


def _overlap_hits(applied_q: torch.Tensor, nq: int, mq: int, n: int, m: int) -> torch.Tensor:
    """applied_q [B][H][W] anchors of an inhibiting rule (n_q x m_q patches); returns
    [B][H][W] > 0 where an n x m patch anchored there overlaps one of those patches."""
    padded = Fn.pad(applied_q[:, None], (mq - 1, m - 1, nq - 1, n - 1))
    ones = torch.ones((1, 1, nq + n - 1, mq + m - 1), dtype=torch.float64)
    return Fn.conv2d(padded, ones)[:, 0]


def step(maps: np.ndarray, rules, actions: np.ndarray, sequential: bool = False,
         control=None, n_step: int = 0, envs=None):
    """One step with one rule list shared by all envs; no episode logic.
    maps uint8 [B][C][H][W]; rules: list of (n, m, I [C+1][n][m], O, reward).
    sequential: each rule's convolution pair is applied (and clamped) before the next rule
    is matched, instead of summing all rules' writes onto the same map.
    control: None or (limit [R], inhibit [R][R], order, seed) for the loaded rules, with
    n_step the batch step number and envs the env indices of the B maps (random keys).
    Returns (maps after, before any reset) uint8, rewards float64 [B]."""
    B, C, H, W = maps.shape
    envs = np.arange(B) if envs is None else envs
    X = torch.zeros((B, C + 1, H, W), dtype=torch.float64)
    X[:, :C] = torch.from_numpy(maps.astype(np.float64))
    X[:, C] = force_plane(X[:, PLAYER], actions)
    delta = torch.zeros_like(X)
    rho = torch.zeros(B, dtype=torch.float64)
    keys = None
    if control is not None:
        keys = [torch.from_numpy(site_keys(control[2], control[3], n_step, int(b), H, W)
                                 .astype(np.float64)).reshape(H, W) for b in envs]
    applied = []              # per loaded rule: [B][H][W] applied anchors
    for idx, (n, m, I, O, rew) in enumerate(move_rules(C) + list(rules)):
        r = idx - 4
        if n > H or m > W:      # no anchor where the pattern lies on the map
            if r >= 0:
                applied.append(torch.zeros((B, H, W), dtype=torch.float64))
            continue
        k_in, thr, k_out = kernels(I[:, :n, :m], O[:, :n, :m])
        act = torch.relu(Fn.conv2d(X, k_in) - thr + 1.0)          # [B][1][H-n+1][W-m+1]
        if control is not None and r >= 0:
            limit, inhibit = control[0], control[1]
            full = torch.zeros((B, H, W), dtype=torch.float64)
            full[:, :H - n + 1, :W - m + 1] = act[:, 0]
            for q in range(r):
                if inhibit[q][r]:
                    nq, mq = rules[q][0], rules[q][1]
                    full[_overlap_hits(applied[q], nq, mq, n, m) > 0] = 0.0
            if limit[r] > 0:
                for bi in range(B):
                    idxs = torch.nonzero(full[bi].flatten()).flatten()
                    if len(idxs) > limit[r]:
                        kv = keys[bi].flatten()[idxs]
                        order = torch.argsort(kv, descending=True)
                        drop = idxs[order[limit[r]:]]
                        full[bi].view(-1)[drop] = 0.0
            applied.append(full)
            act = full[:, None, :H - n + 1, :W - m + 1].contiguous()
        rho += rew * act.sum(dim=(1, 2, 3))
        delta += Fn.conv_transpose2d(act, k_out)                  # [B][C+1][H][W]
        if sequential:
            X = (X + delta >= 1.0).double()
            delta = torch.zeros_like(X)
    Xn = (X + delta >= 1.0)
    return Xn[:, :C].numpy().astype(np.uint8), rho.numpy()


def rules_from_abi(shape, in_pat, out_pat, reward, s: int = 0):
    out = []
    for r in range(shape.shape[1]):
        n, m = int(shape[s, r, 0]), int(shape[s, r, 1])
        out.append((n, m, in_pat[s, r, :, :n, :m], out_pat[s, r, :, :n, :m],
                    int(reward[s, r])))
    return out


def run(maps, rules_abi, actions, L: int = 0, per_env: bool = False, sequential: bool = False,
        control=None):
    """Episode-level stepping on top of `step`: done when no player is left or the counter
    reaches L; done envs return to their initial maps.  Returns per-step maps, rewards,
    done like oracle.run.  control: None or (limit [S][R], inhibit [S][R][R], order, seed)."""

    def ctl(s):
        if control is None:
            return None
        return control[0][s], control[1][s], control[2], control[3]

    shape, in_pat, out_pat, reward = rules_abi
    B = maps.shape[0]
    cur = maps.copy()
    t = np.zeros(B, np.int64)
    T = actions.shape[0]
    out_m = np.zeros((T,) + maps.shape, np.uint8)
    out_r = np.zeros((T, B), np.float32)
    out_d = np.zeros((T, B), np.uint8)
    for k in range(T):
        if per_env:
            nxt = np.zeros_like(cur)
            rho = np.zeros(B)
            for b in range(B):
                nb, rb = step(cur[b:b + 1], rules_from_abi(shape, in_pat, out_pat, reward, b),
                              actions[k, b:b + 1], sequential, ctl(b), k, [b])
                nxt[b], rho[b] = nb[0], rb[0]
        else:
            nxt, rho = step(cur, rules_from_abi(shape, in_pat, out_pat, reward), actions[k],
                            sequential, ctl(0), k)
        t += 1
        done = (nxt[:, PLAYER].reshape(B, -1).sum(1) == 0) | ((L > 0) & (t == L))
        nxt[done] = maps[done]
        t[done] = 0
        cur = nxt
        out_m[k], out_r[k], out_d[k] = cur, rho.astype(np.float32), done
    return out_m, out_r, out_d
