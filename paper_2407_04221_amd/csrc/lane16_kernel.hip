// lane16 step kernel: maps of at most 16 x 16 with one rule set shared by the batch.
//
// This file is the kernel's fixed part.  av_load_rules turns the rule set into straight-line
// bit-sliced code (the body inserted at the RULES marker) and compiles the whole kernel for
// gfx950 with hipRTC; the file also builds on its own, with no rules, as a syntax check.
//
// Layout on chip: a wave's four 16-lane DPP rows each hold one pair of environments; lane y
// of a row holds map row y of both, environment 2p in bits 0-15 and 2p+1 in bits 16-31
// (bit x = column x).  Every plane is one 32-bit register per lane.  Moving a plane up or
// down by i rows is a DPP row shift, fused by the compiler into the consuming VALU op;
// moving it by j columns is a shift of the register.  Rows H..15 and columns W..15 of each
// half are kept zero.
//
// Environments of a wave that do not exist (B not a multiple of 8) compute on zero rows and
// are never stored.  The launch issues all of its first loads (current and initial rows, step
// counters, three blocks of actions) before using any, so it waits for memory once.  The
// initial rows are read by a wave when one of its environments first ends an episode, and
// then stay in registers for later resets.  Actions are read 16 steps at a time and
// turned into per-direction force masks, which each step fetches across its row with
// ds_bpermute one step ahead; rewards and done flags are kept in registers for 16 steps and
// stored together.
//
// One step, per the paper (Sec. 2.1, Sec. 2.1.1, Sec. 2.2.1):
//   force    F = the player plane moved one cell in each environment's action direction;
//   rules    (generated) every rule is matched on the same map: the AND of its specified
//            input entries, each a plane moved by the entry's offset, within the valid-anchor
//            mask; votes of the matches are OR-ed per channel and sign; a wave whose cells
//            got votes of both signs on some channel counts them exactly with carry-save
//            adders; rewards are popcounts of the match masks times the rule rewards;
//   done     no player bit left in the environment's half, or the counter reached L;
//   reset    done environments reload their initial rows.
#ifndef __HIPCC_RTC__
#include <hip/hip_runtime.h>
#endif

/*@DEFINES@*/
#ifndef AV_C
#define AV_C 4
#define AV_H 16
#define AV_W 16
#define AV_L 0
#endif

typedef unsigned int u32;

/*@PHILOX@*/
#ifdef AV_RANDOM_SITES
// The random index channel of rule application control for this lane's row of both
// environments: kb[e * 16 + x] = high 20 bits of the Philox word of cell pos = y * W + x
// (stream 0, generation = batch step number, individual = environment) above 4095 - pos.
__device__ inline void site_keys(u32 *kb, int y, int eA, int eB, bool hasA, bool hasB,
                                 unsigned long long n, unsigned long long seed) {
    if (y >= AV_H) return;
    const int p0 = y * AV_W, p1 = p0 + AV_W;
    for (int e = 0; e < 2; ++e) {
        if (!(e ? hasB : hasA)) continue;
        const unsigned long long env = (unsigned long long)(e ? eB : eA);
        for (int blk = p0 / 8; blk * 8 < p1; ++blk) {
            unsigned int w[8];
            av::philox_words(seed, n, env, 0, (unsigned long long)blk, w);
            for (int j = 0; j < 8; ++j) {
                const int pos = blk * 8 + j;
                if (pos >= p0 && pos < p1) kb[e * 16 + pos - p0] = (w[j] & 0xFFFFF000u) | u32(4095 - pos);
            }
        }
    }
}
#endif

#define AV_PLAYER 2
// lane y <- lane y + i (row shift left), lane y <- lane y - i (row shift right), rotate
#define DPP_SHL(x, i) ((u32)__builtin_amdgcn_update_dpp(0, (int)(x), 0x100 + (i), 0xF, 0xF, true))
#define DPP_SHR(x, i) ((u32)__builtin_amdgcn_update_dpp(0, (int)(x), 0x110 + (i), 0xF, 0xF, true))
#define DPP_ROR(x, i) (__builtin_amdgcn_update_dpp(0, (x), 0x120 + (i), 0xF, 0xF, true))
#define ANY(x) (__builtin_amdgcn_ballot_w64((x) != 0u) != 0ull)
#define COLMASK(k) ((k) >= 16 ? 0xFFFFu : ((1u << (k)) - 1u))
#define BOTH(m) ((m) * 0x10001u)
#define HALF(a, b) (((a) ? 0xFFFFu : 0u) | ((b) ? 0xFFFF0000u : 0u))

extern "C" __global__ void __launch_bounds__(256)
av_lane16_step(unsigned short *__restrict__ state, const unsigned short *__restrict__ init,
               int *__restrict__ tctr, const unsigned char *__restrict__ actions,
               float *__restrict__ rewards, unsigned char *__restrict__ done, int B, int K,
               unsigned long long seed, unsigned long long *__restrict__ nctr,
               unsigned char *__restrict__ obs, int w,
               const unsigned short *__restrict__ gsrc, int gnf, int gA,
               const int *__restrict__ gdepth) {
    const int lane = threadIdx.x & 63;
    // Workgroups are dealt to the GPU's 8 XCDs (each with its own L2) in turn: number them so
    // that each XCD takes one contiguous run of environments, whose result rows share cache
    // lines (a bijection for any grid size).
    const unsigned xg = blockIdx.x, xcd = xg % 8u, xq = gridDim.x / 8u, xr = gridDim.x % 8u;
    const unsigned block = xcd * xq + (xcd < xr ? xcd : xr) + xg / 8u;
    const int wave = int((block * blockDim.x + threadIdx.x) >> 6);
    const int y = lane & 15;
    const int eA = 2 * (wave * 4 + (lane >> 4));
    const int eB = eA + 1;
    const bool hasA = eA < B, hasB = eB < B;
    const bool rowok = y < AV_H;
    const u32 CELL = rowok ? BOTH(COLMASK(AV_W)) : 0u;
    const u32 RT_MASK = CELL & ~BOTH(1u);                      // column 0 receives nothing
    const u32 LF_MASK = CELL & ~BOTH(1u << (AV_W - 1));        // column W-1 receives nothing
    // safe (clamped) environment indices for loads; values of absent envs are masked off
    const int iA = hasA ? eA : 0, iB = hasB ? eB : 0;
    // This wave's copy of the batch step number (steps since the reset, all environments
    // together): read here, stored advanced by K at the end by lane 0.  Waves past the
    // batch's last environment own no copy.
    const bool unit = 8 * wave < B;
    const unsigned long long nbase = unit ? nctr[wave] : 0ull;

#ifdef AV_RANDOM_SITES
    __shared__ u32 kbuf[256 * 32];                  // per lane: the site keys of its row
    u32 *const kb = kbuf + threadIdx.x * 32;
#else
    (void)seed;
#endif
    // Search expansion (gsrc set): environment e starts from row block e / gA of gsrc, laid
    // out [C][gnf][H], with its step counter at gdepth[e / gA]; there are no initial maps to
    // return to (an ended episode is never expanded further).
    // Current rows, and the initial rows for automatic resets, held in registers for the whole
    // launch.
    u32 p[AV_C], q[AV_C];
    const unsigned short *const src = gsrc ? gsrc : state;
    const int sstride = gsrc ? gnf : B;
    const int sA = gsrc ? iA / gA : iA, sB = gsrc ? iB / gA : iB;
    const int yy = rowok ? y : 0;
    const u32 keep = HALF(hasA && rowok, hasB && rowok);

    // Actions arrive 16 steps at a time and become force masks: lane y of a row holds, for
    // step k0 + y of its pair, one mask per direction (up, right, down, left) that is all ones
    // over the columns of each environment whose action is that direction and that can take a
    // force cell from that move (the right / left masks leave out the first / last column, so
    // no bit crosses between the two halves).  A step's four masks are fetched across the row
    // with ds_bpermute during the step before.  Blocks: `cur` the current 16 steps, `nxt` the
    // next 16, `raw` the action bytes of the 16 after those.
    // (the two action bytes are loaded unconditionally, from step 0 past the end and from the
    // clamped environment index for absent environments, and stay untouched until their
    // masks are built 16 steps later, so that no step waits for them; masks of steps past the
    // end are never used and absent environments have no player cell)
    auto raw_block = [&](int k0, u32 &ra, u32 &rb) {
        const int k = k0 + y;
        const unsigned char *row = actions + size_t(k < K ? k : 0) * B;
        ra = u32(row[iA]);
        rb = u32(row[iB]);
    };
    // Every global load the launch starts with is issued before any of them is used, so the
    // prologue waits for memory once: the current rows, the step counters and three blocks
    // of actions.  The initial rows are read at the wave's first reset (a search expansion,
    // which never resets, keeps its current rows instead).
    bool have_init = false;
    u32 slo[AV_C], shi[AV_C];
#pragma unroll
    for (int c = 0; c < AV_C; ++c) {
        slo[c] = u32(src[(size_t(c) * sstride + sA) * AV_H + yy]);
        shi[c] = u32(src[(size_t(c) * sstride + sB) * AV_H + yy]);
    }
    const int *const tsrc = gsrc ? gdepth : tctr;
    int tA = tsrc[sA], tB = tsrc[sB];
    u32 ra0, rb0, ra1, rb1, ra, rb;
    raw_block(0, ra0, rb0);
    raw_block(16, ra1, rb1);
    raw_block(32, ra, rb);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int c = 0; c < AV_C; ++c) {
        p[c] = (slo[c] | (shi[c] << 16)) & keep;
        q[c] = p[c];                            // (replaced at the first reset)
    }
    const u32 COLS = BOTH(COLMASK(AV_W));
    auto dir_masks = [&](u32 aA, u32 aB, u32 *m) {
        m[0] = HALF(aA == 1u, aB == 1u) & COLS;
        m[1] = HALF(aA == 2u, aB == 2u) & COLS & ~BOTH(1u);
        m[2] = HALF(aA == 3u, aB == 3u) & COLS;
        m[3] = HALF(aA == 4u, aB == 4u) & COLS & ~BOTH(1u << (AV_W - 1));
    };
    u32 cur[4], nxt[4], g[4];
    dir_masks(ra0, rb0, cur);
    dir_masks(ra1, rb1, nxt);
    const int src_base = (lane & 48) << 2;
#pragma unroll
    for (int d = 0; d < 4; ++d) g[d] = u32(__builtin_amdgcn_ds_bpermute(src_base, int(cur[d])));
    // Every load above has been consumed except the step counters and the third action
    // block: wait for the vector memory counter here, once, rather than inside the loop.
    __builtin_amdgcn_s_waitcnt(0x0F70);             // vmcnt(0); expcnt, lgkmcnt untouched

    // rewards and done flags of 16 steps: lane y of a row keeps step k0 + y of its pair (zero
    // unless that step paid a reward or ended an episode)
    int rbA = 0, rbB = 0;
    u32 dbuf = 0u;

    // (K >= 1 always: a loop with no entry test keeps the prologue's loads in the first block,
    // where they are issued together, instead of next to their first use in the loop)
    int k = 0;
    do {
        const int s = k & 15;
        // force tiles next to every player cell, toward each environment's action
        u32 F;
        {
            const u32 P = p[AV_PLAYER];
            F = ((DPP_SHL(P, 1) & g[0]) | ((P << 1) & g[1]) | (DPP_SHR(P, 1) & g[2]) |
                 ((P >> 1) & g[3])) & CELL;
        }
        // the next step's masks
        {
            const int s1 = (k + 1) & 15;
            if (s1 == 0) {
#pragma unroll
                for (int d = 0; d < 4; ++d) cur[d] = nxt[d];
                dir_masks(ra, rb, nxt);
                raw_block(k + 33, ra, rb);
            }
#pragma unroll
            for (int d = 0; d < 4; ++d)
                g[d] = u32(__builtin_amdgcn_ds_bpermute(src_base + (s1 << 2), int(cur[d])));
        }

        // per-lane reward sums; `paid`: some rule with a reward matched somewhere in the wave
        // (set by the generated code, only under wave-uniform branches)
        int rA = 0, rB = 0;
        bool paid = false;
#ifdef AV_RANDOM_SITES
        const unsigned long long nstep = nbase + (unsigned long long)k;
        bool keys_ready = false;
#endif
        /*@RULES@*/

        // episode end: any player bit left in each half of this 16-lane row
        u32 o = p[AV_PLAYER];
        o |= (u32)DPP_ROR((int)o, 1);
        o |= (u32)DPP_ROR((int)o, 2);
        o |= (u32)DPP_ROR((int)o, 4);
        o |= (u32)DPP_ROR((int)o, 8);
        tA += 1;
        tB += 1;
        const bool dA = ((o & 0xFFFFu) == 0u) || (AV_L > 0 && tA == AV_L);
        const bool dB = ((o >> 16) == 0u) || (AV_L > 0 && tB == AV_L);

#ifndef AV_NO_REWARD
        // reward: sum of the row's 16 lanes, kept by lane s
        if (paid) {
            rA += DPP_ROR(rA, 1);
            rA += DPP_ROR(rA, 2);
            rA += DPP_ROR(rA, 4);
            rA += DPP_ROR(rA, 8);
            rB += DPP_ROR(rB, 1);
            rB += DPP_ROR(rB, 2);
            rB += DPP_ROR(rB, 4);
            rB += DPP_ROR(rB, 8);
            if (y == s) {
                rbA = rA;
                rbB = rB;
            }
        }
#else
        (void)paid;
#endif
        // automatic reset to the initial map and the step counter; lane s keeps the step's
        // done flags
        if (ANY(u32(dA || dB))) {
            if (dA) tA = 0;
            if (dB) tB = 0;
            if (y == s) dbuf = u32(dA) | (u32(dB) << 1);
            if (!gsrc && !have_init) {          // the initial rows, once
                have_init = true;
#pragma unroll
                for (int c = 0; c < AV_C; ++c) {
                    const u32 lo = u32(init[(size_t(c) * B + iA) * AV_H + yy]);
                    const u32 hi = u32(init[(size_t(c) * B + iB) * AV_H + yy]);
                    q[c] = (lo | (hi << 16)) & keep;
                }
            }
            const u32 dm = HALF(dA, dB);
#pragma unroll
            for (int c = 0; c < AV_C; ++c) p[c] = (q[c] & dm) | (p[c] & ~dm);
        }
        // store 16 steps at once; the buffers then start again from zero (a step without a
        // reward or an ended episode leaves them untouched)
        if (s == 15 || k == K - 1) {
            if (y <= s) {
                const size_t at = size_t(k - s + y) * B;
                if (hasA) {
                    rewards[at + eA] = float(rbA);
                    done[at + eA] = (unsigned char)(dbuf & 1u);
                }
                if (hasB) {
                    rewards[at + eB] = float(rbB);
                    done[at + eB] = (unsigned char)(dbuf >> 1);
                }
            }
            rbA = 0;
            rbB = 0;
            dbuf = 0u;
        }
    } while (++k < K);

#pragma unroll
    for (int c = 0; c < AV_C; ++c) {
        if (hasA && rowok) state[(size_t(c) * B + eA) * AV_H + y] = (unsigned short)(p[c] & 0xFFFFu);
        if (hasB && rowok) state[(size_t(c) * B + eB) * AV_H + y] = (unsigned short)(p[c] >> 16);
    }

    // Observation of the final maps (paper Sec. 2.2.2): for each environment, the w x w window
    // of every channel centred on its first player cell in row-major order, 0 off the map and
    // for environments without a player; obs [B][C][w][w] bytes.  The wave's rows and player
    // cells go through LDS; the windows of the wave's eight environments (contiguous in obs)
    // are built in LDS one window row per lane, at the same offset modulo 16 as their global
    // address, and copied out with aligned 16-byte stores.  Dynamic LDS: four waves x
    // (8 C w^2 + 16) bytes, rounded up to 16.
    if (obs) {
        extern __shared__ __align__(16) unsigned char obuf[];
        __shared__ u32 orow[4][AV_C][64];
        __shared__ int opos[4][8];
        const int wv = threadIdx.x >> 6;
#pragma unroll
        for (int c = 0; c < AV_C; ++c) orow[wv][c][lane] = p[c];
        const u32 P = p[AV_PLAYER];
        u32 pa = (P & 0xFFFFu) ? u32(y << 4) | u32(__ffs(P & 0xFFFFu) - 1) : 0xFFFFu;
        u32 pb = (P >> 16) ? u32(y << 4) | u32(__ffs(P >> 16) - 1) : 0xFFFFu;
        pa = min(pa, (u32)DPP_ROR((int)pa, 1));
        pb = min(pb, (u32)DPP_ROR((int)pb, 1));
        pa = min(pa, (u32)DPP_ROR((int)pa, 2));
        pb = min(pb, (u32)DPP_ROR((int)pb, 2));
        pa = min(pa, (u32)DPP_ROR((int)pa, 4));
        pb = min(pb, (u32)DPP_ROR((int)pb, 4));
        pa = min(pa, (u32)DPP_ROR((int)pa, 8));
        pb = min(pb, (u32)DPP_ROR((int)pb, 8));
        if (y == 0) {
            opos[wv][2 * (lane >> 4)] = int(pa);
            opos[wv][2 * (lane >> 4) + 1] = int(pb);
        }
        __syncthreads();
        const int e0 = 2 * (wave * 4);             // first environment of the wave
        const int nenv = B - e0 < 8 ? B - e0 : 8;
        const int per = AV_C * w * w;
        const int region = (8 * per + 16 + 15) & ~15;
        unsigned char *const wbuf = obuf + wv * region;
        unsigned char *const gdst = obs + size_t(e0 > 0 ? e0 : 0) * per;
        const int shift = int(reinterpret_cast<unsigned long long>(gdst) & 15ull);
        unsigned char *const mine = wbuf + shift;
        const int rows = (nenv > 0 ? nenv : 0) * AV_C * w;
        // window row R = (e * C + c) * w + wy, one per lane, stepping by 64
        int e = lane / (AV_C * w), rem = lane - e * (AV_C * w);
        int c = rem / w, wy = rem - c * w;
        for (int R = lane; R < rows; R += 64) {
            const int pos = opos[wv][e];
            const bool has = pos != 0xFFFF;
            const int yy = (pos >> 4) - w / 2 + wy, x0 = (pos & 15) - w / 2;
            const u32 row = (has && yy >= 0 && yy < AV_H) ? orow[wv][c][(e >> 1) * 16 + yy] : 0u;
            const int half = (e & 1) * 16;
            unsigned char *o = mine + size_t(R) * w;
            for (int wx = 0; wx < w; ++wx) {
                const int xx = x0 + wx;
                o[wx] = (unsigned char)((xx >= 0 && xx < AV_W) ? (row >> (half + xx)) & 1u : 0u);
            }
            wy += 64;
            while (wy >= w) {
                wy -= w;
                if (++c == AV_C) { c = 0; ++e; }
            }
        }
        __syncthreads();
        const int total = rows * w;
        const int head = shift ? (16 - shift < total ? 16 - shift : total) : 0;
        for (int i = lane; i < head; i += 64) gdst[i] = mine[i];
        const int nch = (total - head) / 16;
        for (int k = lane; k < nch; k += 64)
            *reinterpret_cast<uint4 *>(gdst + head + 16 * k) =
                *reinterpret_cast<const uint4 *>(mine + head + 16 * k);
        for (int i = head + 16 * nch + lane; i < total; i += 64) gdst[i] = mine[i];
    }
    if (y == 0) {
        if (hasA) tctr[eA] = tA;
        if (hasB) tctr[eB] = tB;
    }
    if (unit && lane == 0) nctr[wave] = nbase + (unsigned long long)K;
}
