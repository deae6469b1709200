"""The mutation operators written a second way, for pinning the oracle: numpy's own Philox
bit generator (Philox4x64-10) for the random words and vectorised numpy for the rest.
Never imports the oracle or the GPU library."""
import numpy as np

M64 = (1 << 64) - 1


def block(seed, generation, individual, stream, blk):
    """The four 64-bit words of Philox4x64-10 at counter (blk, generation, individual,
    stream), key (seed, 0).  numpy advances the counter before each block, hence - 1."""
    ctr = blk + (generation << 64) + (individual << 128) + (stream << 192)
    return np.random.Philox(key=seed, counter=(ctr - 1) % (1 << 256)).random_raw(4)


def words(seed, generation, individual, stream, count):
    """32-bit words 0 .. count - 1 of one stream (low half of each 64-bit word first)."""
    out = np.zeros(((count + 7) // 8) * 8, np.uint64)
    for blk in range(len(out) // 8):
        w = block(seed, generation, individual, stream, blk)
        out[8 * blk:8 * blk + 8:2] = w & 0xFFFFFFFF
        out[8 * blk + 1:8 * blk + 8:2] = w >> 32
    return out[:count]


def word(seed, generation, individual, stream, idx):
    w = block(seed, generation, individual, stream, idx // 8)[(idx % 8) // 2]
    return int((int(w) >> (32 * (idx % 2))) & 0xFFFFFFFF)


def mutate_maps(maps, m):
    n, C, H, W = maps.shape
    out = (maps != 0).astype(np.uint8).reshape(n, -1)
    chan = np.repeat(np.arange(C), H * W)
    allowed = ((int(m.map_channels) >> chan) & 1).astype(bool)
    for k in range(n):
        u = words(m.seed, m.generation, k, 1, C * H * W)
        out[k] ^= (allowed & (u < m.map_flip_p32)).astype(np.uint8)
    return out.reshape(maps.shape)


def mutate_rules(shape, in_pat, out_pat, reward, m):
    S, R, C1, mh, mw = in_pat.shape
    pats = np.stack([in_pat, out_pat], axis=2).astype(np.int64)    # [S][R][2][C1][mh][mw]
    new = pats.copy()
    rw = reward.astype(np.int64).copy()
    ii = np.arange(mh)[:, None]
    jj = np.arange(mw)[None, :]
    chan_ok = ((int(m.entry_channels) >> np.arange(C1)) & 1).astype(bool)
    span = int(m.reward_hi) - int(m.reward_lo) + 1
    for s in range(S):
        u = words(m.seed, m.generation, s, 2, 2 * R * 2 * C1 * mh * mw)
        decide = (u[0::2] < m.entry_p32).reshape(R, 2, C1, mh, mw)
        pick_hi = (u[1::2] & 1).astype(bool).reshape(R, 2, C1, mh, mw)
        for r in range(R):
            n, mm = shape[s, r]
            inside = (ii < n) & (jj < mm)
            change = decide[r] & inside[None, None] & chan_ok[None, :, None, None]
            old = pats[s, r]
            v = np.where((old == -1) | (old == 0), old, 1)
            lo = np.where(v == -1, 0, -1)
            hi = np.where(v == 1, 0, 1)
            new[s, r] = np.where(change, np.where(pick_hi[r], hi, lo), old)
        ur = words(m.seed, m.generation, s, 3, 2 * R)
        for r in range(R):
            if ur[2 * r] < m.reward_p32:
                rw[s, r] = int(m.reward_lo) + int(ur[2 * r + 1]) % span
    return (new[:, :, 0].astype(np.int8), new[:, :, 1].astype(np.int8), rw.astype(np.int32))
