// rows engine: one environment per wave, map row y in lane y, rules from a per-set program.
//
// A wave of 64 lanes holds one environment.  Lane y owns row y of every plane (the C stored
// channels and the force plane); the planes live in the wave's own LDS as 32-bit rows for
// W <= 32 and 64-bit rows for W <= 64, each plane followed by 16 zero rows, so row y + i of
// any pattern entry is a plain LDS read.  With one wave per workgroup nothing is shared and the
// step loop has no barriers; the four-wave variant for tall maps is described at the kernel.
// The environment's rule program (its own set,
// or the shared one) is read 64 words at a time into a register and taken apart with
// v_readlane; each rule's probe record stays in registers for the whole launch.
//
// Per step (paper Sec. 2.1, Sec. 2.1.1, Sec. 2.2.1), for one batch of all rules (parallel
// mode) or one rule after another (sequential mode):
//   force   F = the player plane moved one cell toward the action;
//   probe   (parallel mode) lane r tests rule r's two rarest input entries together at every
//           anchor row; rules whose probes never hold together are not visited;
//   match   a visited rule ANDs its specified input entries, rarest first, each the plane row
//           y + i shifted right by j (complemented for must-be-0), within the valid-anchor
//           mask, and is left as soon as no anchor of the wave survives;
//   votes   every nonzero K_O = O - I entry (i, j) ORs the match row, shifted left by j, into
//           row y + i of its plane's plus or minus accumulator; the match plane is kept for
//           exact counts;
//   write   new = (old | plus) & ~minus on planes where no cell got both signs; a plane with
//           mixed cells is recounted exactly with bit-sliced counters over the votes of the
//           batch's fired rules: new = (old + #plus > #minus) = (old + sum >= 1);
//   end     reward = sum over fired rules of reward * popcount; done when no player bit is
//           left or the counter reaches L; done environments reload their initial rows.
#include <algorithm>

#include "av_internal.h"

namespace av {
namespace {

constexpr int kPad = 16;              // zero rows around each LDS plane (patterns are <= 16)
// exact counts: a cell gets at most one vote per (rule, i, j), so with the old value at most
// 1 + 4 + 60 x 16 x 16 = 15365 < 2^14 votes of one sign
constexpr int kBits = 14;

__device__ inline bool wave_any(bool p) { return __builtin_amdgcn_ballot_w64(p) != 0ull; }
// Does any lane of group g (lanes g hq .. g hq + hq - 1) hold p?
__device__ inline bool group_any(bool p, int hq, int g) {
    const uint64_t bal = __builtin_amdgcn_ballot_w64(p);
    return hq >= 64 ? bal != 0ull : ((bal >> (g * hq)) & ((1ull << hq) - 1ull)) != 0ull;
}
__device__ inline int popc(uint32_t v) { return __popc(v); }
__device__ inline int popc(uint64_t v) { return __popcll(v); }
__device__ inline void lds_or(uint32_t *p, uint32_t v) { atomicOr(p, v); }
__device__ inline void lds_or(uint64_t *p, uint64_t v) {
    atomicOr(reinterpret_cast<unsigned long long *>(p), static_cast<unsigned long long>(v));
}

template <typename RowT>
__device__ inline RowT low_mask(int bits) {
    return bits >= int(8 * sizeof(RowT)) ? ~RowT(0) : ((RowT(1) << bits) - 1);
}

// Storage type of one packed map row of RB bytes.
template <int RB> struct RowStore;
template <> struct RowStore<2> { using T = uint16_t; };
template <> struct RowStore<4> { using T = uint32_t; };
template <> struct RowStore<8> { using T = uint64_t; };

// Add the one-bit plane t to bits k0.. of the bit-sliced counter cnt; the carry ripples
// only as far as some lane still carries.
template <typename RowT>
__device__ inline void count_add(RowT (&cnt)[kBits], RowT t, int k0) {
#pragma unroll
    for (int k = 0; k < kBits; ++k) {
        if (k < k0) continue;
        if (!wave_any(t != 0)) break;
        const RowT carry = cnt[k] & t;
        cnt[k] ^= t;
        t = carry;
    }
}

// A bit-sliced counter fed one plane at a time: planes are paired, each pair goes into bit
// 0 through one full adder, and only the pair's carry ripples upward.
template <typename RowT>
struct PairCounter {
    RowT cnt[kBits];
    RowT held;
    bool holding;
    __device__ void add(RowT t) {
        if (!holding) {
            held = t;
            holding = true;
            return;
        }
        const RowT a = cnt[0];
        cnt[0] = a ^ held ^ t;
        count_add<RowT>(cnt, (a & held) | (t & (a ^ held)), 1);
        holding = false;
    }
    __device__ void flush() {
        if (holding) count_add<RowT>(cnt, held, 0);
        holding = false;
    }
};

// The rule program of one set, read 64 words at a time: lane l of `v` holds word base + l,
// and a word is taken out of the chunk with v_readlane (a uniform index, no memory access).
// The words come from the set's copy in LDS when it is staged there, else from global memory.
struct Chunk {
    const uint32_t *lds;            // the LDS copy, or null
    const uint32_t *glb;
    int base;
    uint32_t v;
    __device__ void load(int at, int y) {
        base = at;
        v = lds ? lds[at + y] : glb[at + y];   // every set block ends with 64 padding words
    }
    __device__ uint32_t word(int at, int y) {
        if (unsigned(at - base) >= 64u) load(at, y);
        return uint32_t(__builtin_amdgcn_readlane(int(v), at - base));
    }
};

// The test of one input entry (channel, row i, column j, value) at this lane's anchor row:
// plane row ry + i shifted right by j, complemented for a must-be-0 entry.
template <typename RowT>
__device__ inline RowT entry_test(const RowT *Pl, int hp, uint32_t q, int ry) {
    const RowT v = Pl[int(q & 255u) * hp + ry + int((q >> 8) & 255u)] >> int((q >> 16) & 255u);
    return ((q >> 24) & 1u) ? v : RowT(~v);
}

// Exact write of plane c for this lane's row over the rules listed in fired[0..nf) (rule
// index | body offset << 8): every vote on c of every such rule is counted, plus and minus
// separately with the old value as a plus vote, and the cell becomes 1 iff
// old + #plus > #minus.  A rule's votes on c come from its channel index; its match plane
// is slot r of Ms (hs rows, kPad zero rows first).  y: this lane; ry: the row it reads.
template <typename RowT>
__device__ __noinline__ RowT exact_plane(int c, RowT old, const int *fired, int nf,
                                         const uint32_t *lbody, const uint32_t *gbody,
                                         const RowT *Ms, int hs, int y, int ry) {
    PairCounter<RowT> pc, nc;
#pragma unroll
    for (int k = 0; k < kBits; ++k) pc.cnt[k] = nc.cnt[k] = 0;
    pc.cnt[0] = old;
    pc.held = nc.held = 0;
    pc.holding = nc.holding = false;
    for (int f = 0; f < nf; ++f) {
        const int fr = __builtin_amdgcn_readfirstlane(fired[f]);
        const int r = fr & 255, bo = fr >> 8;
        Chunk ch{lbody, gbody, 0, 0u};
        ch.load(bo, y);
        const int cidx = bo + 4 + int(ch.word(bo + 1, y)) + int(ch.word(bo + 2, y));
        const int off = bo + int(ch.word(cidx + 2 * c, y));
        const uint32_t cnts = ch.word(cidx + 2 * c + 1, y);
        const int np = int(cnts & 0xFFFFu), nn = int(cnts >> 16);
        const RowT *Mr = Ms + size_t(r) * hs + kPad + ry;
        for (int e = 0; e < np + nn; ++e) {
            const uint32_t q = ch.word(off + e, y);
            const RowT t = RowT(Mr[-int(q & 255u)] << int(q >> 8));
            if (e < np) pc.add(t);
            else nc.add(t);
        }
    }
    pc.flush();
    nc.flush();
    RowT gt = 0, eq = ~RowT(0);
#pragma unroll
    for (int k = kBits - 1; k >= 0; --k) {
        gt |= eq & pc.cnt[k] & ~nc.cnt[k];
        eq &= ~(pc.cnt[k] ^ nc.cnt[k]);
    }
    return gt;
}

struct RowsArgs {
    const uint32_t *words;   // [S][set_words]: probe records, rule bodies, 64 padding words
    int32_t set_words;
    int32_t rules;           // rules per set (moves included), at most 64
    int32_t body_lds;        // 1: each wave copies its set's words into LDS first
};

// kWaves waves per environment: wave 0 runs the step; with kWaves = 4 (parallel rule order)
// the other three help with the probe pass and the four-entry filter (each wave takes a
// quarter of the anchor rows) and with matching the candidates (each wave takes every fourth
// one, ORs its votes into the shared accumulators and adds its reward, rule count and voted
// planes to three shared counters); wave 0 then writes the planes.  The waves meet at a
// barrier after the force, after the probe, after the filter (when it runs) and after the
// match (when there are candidates).
template <typename RowT, int RB, int kWaves>
__global__ void __launch_bounds__(64 * kWaves) rows_step(StepArgs a, RowsArgs rp) {
    using ST = typename RowStore<RB>::T;
    extern __shared__ __align__(16) unsigned char lds[];
    const int Rt = rp.rules;
    constexpr int nw = kWaves;
    const int y = int(threadIdx.x & 63u);
    const int wv = nw == 1 ? 0 : __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int b = int(blockIdx.x);
    const int H = a.H, W = a.W, C = a.C, B = a.B;
    const int hp = H + kPad;          // rows per LDS plane
    const bool row = y < H;
    const int ry = row ? y : 0;       // a row that is safe to address for idle lanes
    RowT *Pl = reinterpret_cast<RowT *>(lds);              // [C + 2][hp]: planes, F, zeros
    RowT *Vp = Pl + size_t(C + 2) * hp;                    // [C + 1][hp]: plus votes
    RowT *Vm = Vp + size_t(C + 1) * hp;                    // [C + 1][hp]: minus votes
    RowT *Ms = Vm + size_t(C + 1) * hp;                    // [Rt][kPad + hp]: match planes
    const int hs = kPad + hp;
    int *fired = reinterpret_cast<int *>(Ms + size_t(Rt) * hs);   // [Rt]
    uint32_t *prob = reinterpret_cast<uint32_t *>(fired + Rt);     // [8 Rt] probe records
    uint32_t *tslot = prob + 8 * Rt;                                // [4][2]: waves' candidates
    uint32_t *tfilt = tslot + 8;                                    // [4][2]: after the filter
    int *lcnt = reinterpret_cast<int *>(tfilt + 8);   // fired rules, voted planes, reward
    uint32_t *lprog = tslot + 24;                                   // [set_words] if staged
    const uint32_t *gprog = rp.words + size_t(a.per_env ? b : 0) * size_t(rp.set_words);
    const RowT wmask = low_mask<RowT>(W);
    // row y of environment b in channel c is element c * plane + lrow of the [C][B][H] arrays
    const size_t plane = size_t(B) * H;
    const size_t lrow = size_t(b) * H + size_t(ry);

    // zero: the planes with their pad rows, the vote accumulators, and the pad rows above
    // every match plane (the rows below them are written before they are read)
    const int pwords = int(size_t(3 * C + 4) * hp * (sizeof(RowT) / 4));
    if (wv == 0) {
        for (int w = y; w < pwords; w += 64) reinterpret_cast<uint32_t *>(lds)[w] = 0u;
        for (int w = y; w < Rt * kPad; w += 64) Ms[size_t(w / kPad) * hs + (w % kPad)] = 0;
        for (int w = y; w < 8 * Rt; w += 64) prob[w] = gprog[w];
        if (rp.body_lds)
            for (int w = y; w < rp.set_words; w += 64) lprog[w] = gprog[w];
    }
    const uint32_t *const lbody = rp.body_lds ? lprog : nullptr;
    // probe records (8 words per rule): lane l of pt[g] holds word 64 g + l, i.e. word l % 8
    // of rule 8 g + l / 8
    uint32_t pt[8];
#pragma unroll
    for (int g = 0; g < 8; ++g) pt[g] = (64 * g + y < 8 * Rt) ? gprog[64 * g + y] : 0u;
    // Lane-parallel probes (parallel rule order): lane r tests the first two (or, on a
    // second pass, four) entries of rule r's rarest-first list together at every anchor row;
    // a missing entry reads the zero plane C + 1 complemented, which passes everywhere.
    int pa[4], pj[4], pmax = -1;
    RowT pinv[4], pcol = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        pa[e] = (C + 1) * hp;
        pj[e] = 0;
        pinv[e] = ~RowT(0);
    }
    if (y < Rt) {
        const uint32_t *rec = gprog + 8 * y;
        const uint32_t w0 = rec[0];
        const int n = int(w0 & 255u), m = int((w0 >> 8) & 255u);
        const int ecnt = int(rec[4]);
        const uint32_t first[4] = {rec[1], rec[2], rec[5], rec[6]};
        pmax = H - n;
        pcol = low_mask<RowT>(W - m + 1);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (e < ecnt) {
                const uint32_t q = first[e];
                pa[e] = int(q & 255u) * hp + int((q >> 8) & 255u);
                pj[e] = int((q >> 16) & 255u);
                pinv[e] = ((q >> 24) & 1u) ? RowT(0) : ~RowT(0);
            }
    }
    __syncthreads();
    if (wv == 0)
        for (int c = 0; c < C; ++c)
            if (row) Pl[c * hp + y] = RowT(static_cast<const ST *>(a.state)[c * plane + lrow]);
    // this wave's share of the probe pass's anchor rows
    const int y0 = wv * H / nw, y1 = (wv + 1) * H / nw;

    int t_env = a.t[b];
    uint32_t ablk = 0;
    float rbuf = 0.f;     // lane l: reward of step k0 + l of the current block of 64 steps
    uint32_t dbuf = 0;    // lane l: done flag of that step
    const uint64_t all_rules = Rt >= 64 ? ~0ull : ((1ull << Rt) - 1ull);
    RowT *const F = Pl + size_t(C) * hp;
    const RowT *const P = Pl + size_t(kChPlayer) * hp;

    for (int k = 0; k < a.k; ++k) {
        if (wv == 0) {
        // actions come 64 steps at a time: lane l holds step k0 + l
        if ((k & 63) == 0) ablk = (k + y < a.k) ? uint32_t(a.actions[size_t(k + y) * B + b]) : 0u;
        const int act = __builtin_amdgcn_readlane(int(ablk), k & 63);
        {
            RowT f = 0;
            if (act == 1) f = P[ry + 1];                    // row H is a zero pad row
            else if (act == 3) f = ry > 0 ? P[ry - 1] : RowT(0);
            else if (act == 2) f = (P[ry] << 1) & wmask;
            else if (act == 4) f = P[ry] >> 1;
            if (row) F[y] = f;
        }
        if (nw > 1 && y < 3) lcnt[y] = 0;
        }
        if (nw > 1) __syncthreads();             // the map and this step's force plane are set
        int rsum = 0, nf = 0;
        uint32_t touched = 0;   // planes that received votes in the current batch
        // The rules to visit: in sequential order every rule, one batch each (each matches the
        // map the rules before it left); in parallel order the candidates, one batch: rules
        // whose two probes hold together at some anchor (lane r tests rule r).
        uint64_t todo = all_rules;
        if (!a.sequential) {
            RowT hit = 0;
            for (int yy = y0; yy < y1; ++yy) {
                const RowT t = ((Pl[pa[0] + yy] >> pj[0]) ^ pinv[0]) &
                               ((Pl[pa[1] + yy] >> pj[1]) ^ pinv[1]);
                hit |= yy <= pmax ? t : RowT(0);
            }
            todo = __builtin_amdgcn_ballot_w64((hit & pcol) != 0);
            if (nw > 1) {
                // the waves' candidates, OR-ed (wave 0 reads the slots before the next step)
                if (y == 0) {
                    tslot[2 * wv] = uint32_t(todo);
                    tslot[2 * wv + 1] = uint32_t(todo >> 32);
                }
                __syncthreads();
                todo = 0;
                for (int w = 0; w < nw; ++w)
                    todo |= uint64_t(tslot[2 * w]) | (uint64_t(tslot[2 * w + 1]) << 32);
            }
        }
        if (!a.sequential) {
            if (__popcll(todo) > 2) {
                // many candidates (crowded maps): filter them with four entries at once
                RowT hit = 0;
                for (int yy = nw > 1 ? y0 : 0; yy < (nw > 1 ? y1 : H); ++yy) {
                    const RowT t = ((Pl[pa[0] + yy] >> pj[0]) ^ pinv[0]) &
                                   ((Pl[pa[1] + yy] >> pj[1]) ^ pinv[1]) &
                                   ((Pl[pa[2] + yy] >> pj[2]) ^ pinv[2]) &
                                   ((Pl[pa[3] + yy] >> pj[3]) ^ pinv[3]);
                    hit |= yy <= pmax ? t : RowT(0);
                }
                uint64_t keep = __builtin_amdgcn_ballot_w64((hit & pcol) != 0);
                if (nw > 1) {
                    if (y == 0) {
                        tfilt[2 * wv] = uint32_t(keep);
                        tfilt[2 * wv + 1] = uint32_t(keep >> 32);
                    }
                    __syncthreads();
                    keep = 0;
                    for (int w = 0; w < nw; ++w)
                        keep |= uint64_t(tfilt[2 * w]) | (uint64_t(tfilt[2 * w + 1]) << 32);
                }
                todo &= keep;
            }
            if (nw == 1 && H <= 32 && __popcll(todo) > 2) {
                // Several candidates on a map of at most 32 rows: the wave splits into groups
                // of hq lanes (lane gy of a group on map row gy) that match one candidate each
                // at the same time.  A group reads its rule's entries and votes from its own
                // hq-word chunk of the program (lane gy holds word base + gy, taken out with
                // ds_bpermute) and leaves the rule when none of its anchors survives.
                const int hq = H <= 16 ? 16 : 32, G = 64 / hq;
                const int g = y / hq, gy = y - g * hq;
                const bool grow = gy < H;
                const int gry = grow ? gy : 0;
                const uint32_t *const body = lbody ? lbody : gprog;
                uint32_t tmask = 0;
                while (todo) {
                    int rsel = -1;
                    for (int q = 0; q < G && todo; ++q) {
                        const int r = int(__builtin_ctzll(todo));
                        todo &= todo - 1ull;
                        if (g == q) rsel = r;
                    }
                    const bool mine = rsel >= 0;
                    const int rr = mine ? rsel : 0;
                    const uint32_t w0 = prob[8 * rr];
                    const int bo = int(prob[8 * rr + 3]);
                    const int n = int(w0 & 255u), m = int((w0 >> 8) & 255u);
                    const uint32_t *const bp = body + bo;
                    const int reward = int(bp[0]), ecnt = mine ? int(bp[1]) : 0;
                    const int vcnt = int(bp[2]);
                    RowT M = (mine && gy + n <= H) ? low_mask<RowT>(W - m + 1) : RowT(0);
                    bool alive = mine;
                    int cb = 0;
                    uint32_t cv = bp[4 + gy];          // every set block ends with 64 zero words
                    for (int e = 0; wave_any(alive && e < ecnt);) {
                        if (e - cb >= hq) {
                            cb = e;
                            cv = bp[4 + cb + gy];
                        }
                        const int lim = min(e == 0 ? 2 : 4, cb + hq - e);
                        for (int u = 0; u < lim; ++u) {
                            const uint32_t q = uint32_t(__builtin_amdgcn_ds_bpermute(
                                (g * hq + e + u - cb) << 2, int(cv)));
                            if (e + u < ecnt) M &= entry_test<RowT>(Pl, hp, q, gry);
                        }
                        e += lim;
                        alive = group_any(M != 0, hq, g);
                    }
                    const bool hit = mine && group_any(M != 0, hq, g);
                    if (hit) {
                        if (grow) Ms[size_t(rr) * hs + kPad + gy] = M;
                        rsum += reward * popc(M);
                    }
                    cb = 0;
                    cv = bp[4 + ecnt + gy];
                    for (int v = 0; wave_any(hit && v < vcnt); ++v) {
                        if (v - cb >= hq) {
                            cb = v;
                            cv = bp[4 + ecnt + cb + gy];
                        }
                        const uint32_t q = uint32_t(__builtin_amdgcn_ds_bpermute(
                            (g * hq + v - cb) << 2, int(cv)));
                        if (hit && v < vcnt && grow) {
                            const int c = int(q & 255u), i = int((q >> 8) & 255u);
                            const int j = int((q >> 16) & 255u);
                            lds_or((((q >> 24) & 1u) ? Vp : Vm) + c * hp + gy + i, RowT(M << j));
                            tmask |= 1u << c;
                        }
                    }
                    // record the rules that fired (rule index | body offset << 8)
                    const uint64_t hits = __builtin_amdgcn_ballot_w64(hit);
                    for (int q = 0; q < G; ++q)
                        if ((hits >> (q * hq)) & 1ull) {
                            const int rq = __builtin_amdgcn_readlane(rsel, q * hq);
                            const int bq = __builtin_amdgcn_readlane(bo, q * hq);
                            if (y == 0) fired[nf] = rq | (bq << 8);
                            ++nf;
                        }
                }
                for (int off = 1; off < 64; off <<= 1) tmask |= uint32_t(__shfl_xor(int(tmask), off, 64));
                touched |= uint32_t(__builtin_amdgcn_readfirstlane(int(tmask)));
            }
        }
        // with helper waves and two or more candidates, wave w matches every nw-th candidate
        // from the w-th on (a lone candidate is wave 0's, without meeting the others)
        const bool shared = nw > 1 && (todo & (todo - 1ull)) != 0ull;
        if (shared) {
            uint64_t mine = 0;
            int q = 0;
            for (uint64_t t = todo; t; t &= t - 1ull, ++q)
                if ((q & (nw - 1)) == wv) mine |= t & (0ull - t);
            todo = mine;
        } else if (wv != 0) {
            todo = 0ull;
        }
        for (;;) {
            const bool last = todo == 0ull;
            do {
                if (last) break;
                // match rule r; if it fires, record it, pay its reward and OR its votes
                const int r = int(__builtin_ctzll(todo));
                todo &= todo - 1ull;
                const uint32_t ptr = pt[r >> 3];
                const int lb = (r & 7) * 8;
                const uint32_t w0 = uint32_t(__builtin_amdgcn_readlane(int(ptr), lb));
                const int n = int(w0 & 255u), m = int((w0 >> 8) & 255u);
                const int bo = __builtin_amdgcn_readlane(int(ptr), lb + 3);
                Chunk ch{lbody, gprog, 0, 0u};
                ch.load(bo, y);
                const int reward = int(ch.word(bo, y)), ecnt = int(ch.word(bo + 1, y));
                const int vcnt = int(ch.word(bo + 2, y));
                // entries rarest first, two, then four at a time, leaving the rule as soon as
                // no anchor of the wave survives
                RowT M = (y + n <= H) ? low_mask<RowT>(W - m + 1) : RowT(0);
                bool alive = true;
                for (int e = 0; e < ecnt && alive;) {
                    const int stop = e == 0 ? 2 : e + 4;
                    for (; e < ecnt && e < stop; ++e) M &= entry_test<RowT>(Pl, hp, ch.word(bo + 4 + e, y), ry);
                    alive = wave_any(M != 0);
                }
                if (!alive || !wave_any(M != 0)) break;

                if (row) Ms[size_t(r) * hs + kPad + y] = M;
                if (y == 0) fired[shared ? atomicAdd(&lcnt[0], 1) : nf] = r | (bo << 8);
                ++nf;
                rsum += reward * popc(M);
                // votes: the match row, shifted left by j, into row y + i of the accumulator
                const int voff = bo + 4 + ecnt;
                for (int e = 0; e < vcnt; ++e) {
                    const uint32_t q = ch.word(voff + e, y);
                    const int c = int(q & 255u), i = int((q >> 8) & 255u), j = int((q >> 16) & 255u);
                    RowT *acc = ((q >> 24) & 1u) ? Vp : Vm;
                    if (row) lds_or(acc + c * hp + y + i, RowT(M << j));
                    touched |= 1u << c;
                }
            } while (false);
            if (shared && last) {
                // the helper waves add their rewards and voted planes to the shared counters;
                // wave 0 goes on with the totals (its own rewards stay in its lanes)
                if (wv != 0) {
                    if (wave_any(rsum != 0))
                        for (int off = 32; off > 0; off >>= 1) rsum += __shfl_xor(rsum, off, 64);
                    if (y == 0) {
                        if (rsum != 0) atomicAdd(&lcnt[2], rsum);
                        if (touched != 0) atomicOr(reinterpret_cast<unsigned *>(&lcnt[1]), touched);
                    }
                }
                __syncthreads();
                if (wv != 0) break;
                nf = lcnt[0];
                touched |= uint32_t(lcnt[1]);
                if (y == 0) rsum += lcnt[2];
            }
            if (nf > 0 && (a.sequential || last)) {
                // write the planes the batch's rules voted on; planes where some cell got
                // votes of both signs are recounted exactly
                for (uint32_t t = touched; t; t &= t - 1) {
                    const int c = __builtin_ctz(t);
                    const RowT old = Pl[c * hp + ry], pl = Vp[c * hp + ry], mi = Vm[c * hp + ry];
                    RowT nv = (old | pl) & ~mi;
                    if (wave_any((pl & mi) != 0))
                        nv = exact_plane<RowT>(c, old, fired, nf, lbody, gprog, Ms, hs, y, ry);
                    if (row) {
                        Pl[c * hp + y] = nv;
                        Vp[c * hp + y] = 0;
                        Vm[c * hp + y] = 0;
                    }
                }
                touched = 0;
                nf = 0;
            }
            if (last) break;
        }
        if (wv != 0) continue;                    // helper waves: the rest is wave 0's

        // reward: wave sum of the lanes' counts
        int total = 0;
        if (wave_any(rsum != 0)) {
            for (int off = 32; off > 0; off >>= 1) rsum += __shfl_xor(rsum, off, 64);
            total = rsum;
        }
        const bool anyp = wave_any(row && P[y] != 0);
        t_env += 1;
        const bool d = !anyp || (a.L > 0 && t_env == a.L);
        if (d) t_env = 0;
        if (y == (k & 63)) {
            rbuf = float(total);
            dbuf = d ? 1u : 0u;
        }
        if ((k & 63) == 63 || k == a.k - 1) {
            const int k0 = k & ~63;
            if (y <= (k & 63)) {
                a.rewards[size_t(k0 + y) * B + b] = rbuf;
                a.done[size_t(k0 + y) * B + b] = uint8_t(dbuf);
            }
        }
        if (d)
            for (int c = 0; c < C; ++c)
                if (row) Pl[c * hp + y] = RowT(static_cast<const ST *>(a.init)[c * plane + lrow]);
    }

    if (wv != 0) return;
    for (int c = 0; c < C; ++c)
        if (row) static_cast<ST *>(a.state)[c * plane + lrow] = ST(Pl[c * hp + y]);
    if (y == 0) {
        a.t[b] = t_env;
        a.nctr[b] += uint64_t(a.k);     // the batch step number (no rule control here)
    }
}

}  // namespace

// ---------------------------------------------------------------------------------
// Host side: the rows program, one block of words per rule set, built from the generic
// program.  Block layout (word offsets from the block start):
//   [8 r, 8 r + 8)  probe record of rule r: n | m << 8 | probes << 16, its first two
//                   entries rarest first (0 if fewer), the body offset, the entry count,
//                   its third and fourth entries, 0
//   body of rule r: reward, entry count, vote count, 0; every specified entry, rarest
//                   first; the votes; per channel c of C + 1 two words: the offset (from the
//                   body start) of c's votes and their counts (plus | minus << 16); those
//                   votes, plus then minus, as i | j << 8
//   64 zero words   so that a 64-word chunk read never leaves the block
// Entry and vote words use the generic encodings (channel, i, j, value / sign).
// "Rarest first" orders entries by the share of cells they accept on a typical map:
// must-be-1 on force or player (about 1 cell), on goal or extra tiles (a fifth), on wall
// (under a third), on empty; then must-be-0 on the same channels in the reverse order
// (must-be-0 on force or player accepts almost every cell).
// ---------------------------------------------------------------------------------
namespace {
int accept_rank(uint32_t q, int C) {
    const int c = int(q & 255u), want = int((q >> 24) & 1u);
    int ch;
    if (c == C) ch = 0;
    else if (c == kChPlayer) ch = 1;
    else if (c == kChGoal || c >= 4) ch = 2;
    else if (c == kChWall) ch = 3;
    else ch = 4;
    return want ? ch : 10 - ch;
}
}  // namespace

void compile_rows(const GenericProgram &g, int C, RowsProgram &out) {
    const int Rt = g.rules_per_set, S = g.sets;
    std::vector<std::vector<uint32_t>> sets(S);
    for (int s = 0; s < S; ++s) {
        std::vector<uint32_t> &w = sets[s];
        w.assign(size_t(Rt) * 8, 0);
        for (int r = 0; r < Rt; ++r) {
            const RuleHdr &h = g.hdr[size_t(s) * Rt + r];
            const uint32_t *ms = g.match.data() + size_t(s) * g.match_stride + h.match_off;
            const uint32_t *vs = g.rvote.data() + size_t(s) * g.rvote_stride + h.vote_off;
            std::vector<uint32_t> ents(ms, ms + h.match_cnt);
            std::stable_sort(ents.begin(), ents.end(), [C](uint32_t a, uint32_t b) {
                return accept_rank(a, C) < accept_rank(b, C);
            });
            const std::vector<uint32_t> votes(vs, vs + h.vote_cnt);
            const int probes = std::min(2, h.match_cnt);
            const size_t body = w.size();
            uint32_t *rec = &w[size_t(r) * 8];
            rec[0] = uint32_t(h.n) | (uint32_t(h.m) << 8) | (uint32_t(probes) << 16);
            rec[1] = probes > 0 ? ents[0] : 0u;
            rec[2] = probes > 1 ? ents[1] : 0u;
            rec[3] = uint32_t(body);
            rec[4] = uint32_t(ents.size());
            rec[5] = ents.size() > 2 ? ents[2] : 0u;
            rec[6] = ents.size() > 3 ? ents[3] : 0u;
            w.push_back(uint32_t(h.reward));
            w.push_back(uint32_t(ents.size()));
            w.push_back(uint32_t(votes.size()));
            w.push_back(0u);
            w.insert(w.end(), ents.begin(), ents.end());
            w.insert(w.end(), votes.begin(), votes.end());
            const size_t index = w.size();
            w.insert(w.end(), size_t(2) * (C + 1), 0u);
            for (int c = 0; c <= C; ++c) {
                uint32_t np = 0, nn = 0;
                w[index + 2 * c] = uint32_t(w.size() - body);
                for (int sign = 1; sign >= 0; --sign)
                    for (uint32_t v : votes)
                        if (int(v & 255u) == c && int((v >> 24) & 1u) == sign) {
                            w.push_back(((v >> 8) & 255u) | (((v >> 16) & 255u) << 8));
                            (sign ? np : nn) += 1;
                        }
                w[index + 2 * c + 1] = np | (nn << 16);
            }
        }
        w.insert(w.end(), 64, 0u);
    }
    out.rules = Rt;
    out.sets = S;
    out.set_words = 1;
    for (auto &w : sets) out.set_words = std::max(out.set_words, int(w.size()));
    out.set_words = (out.set_words + 3) & ~3;
    out.words.assign(size_t(S) * out.set_words, 0);
    for (int s = 0; s < S; ++s) std::copy(sets[s].begin(), sets[s].end(),
                                          out.words.begin() + size_t(s) * out.set_words);
}

// LDS of one wave: C + 2 planes, 2 (C + 1) vote accumulators and one match plane per rule
// (H + 16 rows each, the match planes 16 more), the fired list and the probe records.
size_t rows_lds_bytes(int H, int W, int C, int rules_per_set) {
    const size_t rowb = W <= 32 ? 4 : 8, hp = size_t(H) + kPad;
    return ((size_t(C + 2) + size_t(2) * (C + 1)) * hp + size_t(rules_per_set) * (hp + kPad)) *
               rowb +
           (sizeof(int) + 8 * sizeof(uint32_t)) * size_t(rules_per_set) + 24 * sizeof(uint32_t);
}

bool rows_eligible(int H, int W, int C, int rules_per_set) {
    return H <= 64 && W <= 64 && C <= 31 && rules_per_set <= 64 &&
           rows_lds_bytes(H, W, C, rules_per_set) <= size_t(kLdsBudget);
}

hipError_t launch_rows_step(const StepArgs &a, const uint32_t *words, int set_words, int rules,
                            hipStream_t s) {
    if (!rows_eligible(a.H, a.W, a.C, rules)) return hipErrorInvalidValue;
    size_t lds = rows_lds_bytes(a.H, a.W, a.C, rules);
    // Stage the program in LDS for launches of 16 steps or more, when it fits and does not
    // cost occupancy: with more than one
    // workgroup per CU to place (256 CUs, 160 KiB of LDS each), the staged wave must still
    // leave room for its share of them.
    const size_t staged = lds + sizeof(uint32_t) * size_t(set_words);
    const size_t per_cu = (size_t(a.B) + 255) / 256;
    const int body_lds = a.k >= 16 && staged <= size_t(kLdsBudget) &&
                         staged * per_cu <= size_t(160) * 1024;
    if (body_lds) lds = staged;
    // On maps taller than 32 rows the probe pass (a loop over every anchor row) is most of a
    // step, and a crowded map has many candidates to match one after another; when the batch
    // leaves the wave slots for it, three more waves per environment take three quarters of
    // the probe's rows and of the candidates.
    const bool helpers = a.H > 32 && !a.sequential && 4LL * a.B <= device_wave_slots();
    RowsArgs rp{words, set_words, rules, body_lds};
    // (built for 4- and 8-byte rows; maps of at most 16 columns keep one wave)
    if (a.row_bytes == 2)
        hipLaunchKernelGGL((rows_step<uint32_t, 2, 1>), dim3(a.B), dim3(64), lds, s, a, rp);
    else if (a.row_bytes == 4 && !helpers)
        hipLaunchKernelGGL((rows_step<uint32_t, 4, 1>), dim3(a.B), dim3(64), lds, s, a, rp);
    else if (a.row_bytes == 4)
        hipLaunchKernelGGL((rows_step<uint32_t, 4, 4>), dim3(a.B), dim3(256), lds, s, a, rp);
    else if (!helpers)
        hipLaunchKernelGGL((rows_step<uint64_t, 8, 1>), dim3(a.B), dim3(64), lds, s, a, rp);
    else
        hipLaunchKernelGGL((rows_step<uint64_t, 8, 4>), dim3(a.B), dim3(256), lds, s, a, rp);
    return hipGetLastError();
}

}  // namespace av
