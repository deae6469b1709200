// group engine: one environment per wave, its rules dealt to groups of lanes.
//
// The wave's 64 lanes form G = 4 groups of 16 lanes; lane y of every group owns map row y (a
// 32-bit word, bit x = column x) and, on maps of 17 to 32 rows, row y + 16 too (HR = 16 or 32
// rows a group covers), and group g matches rules g, g + G, g + 2G, ...  One workgroup is one
// wave, so a step needs no barrier: the wave's LDS operations take effect in the order it issues
// them.
//
// The four built-in moves are computed in registers from the lanes' own rows of the player,
// wall and force planes and the rows next to them (DPP row shifts within the 16-lane groups;
// with two rows a lane, the rows 15 and 16 meet across the lanes' two words); the player and
// wall rows stay in registers from step to step unless a loaded rule wrote those planes.  A rule's input entries are merged per plane
// row (one LDS read tests every specified column of a pattern row, up to 8); each loaded
// rule's first four merged entries sit in a probe table (held in registers for the launch when
// a group has at most two rules, else read at the start of each step), so the probe of every
// loaded rule is one round of LDS reads with no branch between the rules; only rules that
// pass it somewhere read the rest of their entries, and only channels that received votes are
// rewritten.
//
// LDS (32-bit rows):
//   P    [C+1][PR]     the map and the force plane (channel C); PR = HR + ph - 1 rounded up to
//                      4 rows (ph: the largest pattern's rows), so a lane reads row y + i of
//                      any pattern entry without a bounds test (rows H .. PR - 1 stay zero)
//   M    [R+4][PR]     match planes of the rules that fired, row y at ph - 1 + y: the zero rows
//                      above let a vote read match row y - i without a test
//   PL, MI [C][HR]     per stored channel, the OR of the +1 and of the -1 votes
//   I0   [C][HR]       the initial rows, for resets
//   PT   [R+5][12]     probe table: per loaded rule its first eight merged entries, its
//                      anchor rows and columns, where its entries and its votes are and the
//                      channels it votes on (row R + 4: zeros,
//                      read by groups with fewer rules than others)
//   RS   [C][R+4]      per channel and rule, the range of the rule's votes in the channel's
//                      vote list (for exact recounts)
//   RM   [C][2]        per channel, the 64-bit mask of the rules with votes in that list
//   program            (when it fits, see the launcher) the environment's rule headers, input
//                      merged entries, rule-major votes and channel-major vote lists
//
// Per step (paper Sec. 2.1, Sec. 2.1.1, Sec. 2.2.1):
//   force  F[y] = the player row moved one cell toward the action (group 0 writes it);
//   moves  right P & (F >> 1) & ~(W >> 1), left F & ~W & (P >> 1), down P & F' & ~W', up
//          F & ~W & P' (primes: the next row); their votes on the player plane are OR-ed in
//          registers (-1 on the source cell, +1 on the target);
//   match  per loaded rule, AND over its specified entries of plane row y + i shifted right by j,
//          complemented for must-be-0, within the valid-anchor mask (the entries of one plane
//          row i share its LDS read); a group leaves a rule as soon as no lane of the group has
//          an anchor left;
//   votes  a rule that fired stores its match plane and ORs match row y - i, shifted left by
//          j, into the plus or minus row of each nonzero K_O = O - I entry's channel;
//   write  group g rewrites channels g, g + G, ...: new = (old | plus) & ~minus where no cell
//          got votes of both signs; a channel with such cells is recounted exactly with one
//          bit-sliced counter over every fired rule's votes: new = (old + #plus > #minus);
//   end    done when no player bit is left or the counter reaches L; reward = sum over fired
//          rules of reward * popcount; done environments return to their initial rows.
// Parallel rule order only, without rule application control.
#include <algorithm>
#include <type_traits>

#include "av_internal.h"

namespace av {
namespace {

constexpr int kMaxRulesPerGroup = 16;   // loaded and built-in rules per group, at most
constexpr int kMaxChanPerGroup = 8;     // stored channels a group writes, at most
constexpr int kCountBits = 8;           // exact write counters: a channel list holds <= 254
                                        // entries (eligibility: rules x pattern cells <= 254)
constexpr int kHdrWords = int(sizeof(RuleHdr) / 4);
constexpr int kProbeEntries = 4;        // input entries of every rule tested in one round
constexpr int kProbeWords = 12;         // probe table row: entries 0-3, anchor word, match
                                        // offset | count << 16, vote offset | count << 16,
                                        // voted channels, entries 4-7
// Input entries merged per plane row: o | jb << 12 | care << 16 | want << 24 tests row
// o + y of the planes (o = c * PR + i: pattern row i of plane c) at the pattern columns
// 8 jb + j, j < 8, whose bit j of care is set: there the cell must equal bit j of want.
// kPassEntry tests no column (it passes everywhere).
constexpr uint32_t kPassEntry = 0u;
constexpr int kMaxEntryOffset = 4095;
constexpr int kShortLaunch = 16;        // launches of fewer steps: SHORT kernels, program in
                                        // global memory

// Words per plane row block: HR rows plus the pattern rows hanging below the last one,
// rounded up to 4 (16-byte aligned probe table after the planes).
__host__ __device__ constexpr int group_plane_words(int Hq, int max_pat_h) {
    return (Hq + max_pat_h - 1 + 3) & ~3;
}

__device__ inline uint32_t low_mask(int bits) { return bits >= 32 ? ~0u : ((1u << bits) - 1u); }

// Copy n words from global memory to LDS, eight loads of a lane in flight before its writes.
__device__ inline void copy_to_lds(uint32_t *dst, const uint32_t *src, int n, int lane) {
    for (int w0 = lane; w0 < n; w0 += 8 * 64) {
        uint32_t v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int w = w0 + 64 * u;
            v[u] = w < n ? src[w] : 0u;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int w = w0 + 64 * u;
            if (w < n) dst[w] = v[u];
        }
    }
}

// Does any lane of this lane's group hold a nonzero?
template <int Hq>
__device__ inline bool group_any(bool p, int lane) {
    const unsigned long long bal = __builtin_amdgcn_ballot_w64(p);
    if (Hq >= 64) return bal != 0ull;
    const int base = lane & ~(Hq - 1);
    return ((bal >> base) & ((1ull << Hq) - 1ull)) != 0ull;
}

// Rows y + 1 (next) and y - 1 (prev) of the rows a lane holds, 0 past the group's ends, RPL
// of them (2: on maps of 17 to 32 rows a lane of a 16-lane group holds rows y and y + 16):
// within each 16-row half a DPP row shift, across the halves a DPP row rotate (lane 15's next
// row is lane 0's second row, lane 0's second row's previous row is lane 15's first).
template <int Hq, int RPL>
__device__ inline void next_rows(const uint32_t (&v)[RPL], uint32_t (&n)[RPL], int lane, int y) {
    static_assert(Hq == 16, "16-lane groups");
    (void)lane;
    if constexpr (RPL == 1) {
        n[0] = uint32_t(__builtin_amdgcn_update_dpp(0, int(v[0]), 0x101, 0xF, 0xF, true));
    } else {
        const uint32_t s0 = uint32_t(__builtin_amdgcn_update_dpp(0, int(v[0]), 0x101, 0xF, 0xF, true));
        const uint32_t w1 = uint32_t(__builtin_amdgcn_update_dpp(0, int(v[1]), 0x12F, 0xF, 0xF, true));
        n[0] = y == Hq - 1 ? w1 : s0;
        n[1] = uint32_t(__builtin_amdgcn_update_dpp(0, int(v[1]), 0x101, 0xF, 0xF, true));
    }
}
template <int Hq, int RPL>
__device__ inline void prev_rows(const uint32_t (&v)[RPL], uint32_t (&p)[RPL], int lane, int y) {
    static_assert(Hq == 16, "16-lane groups");
    (void)lane;
    if constexpr (RPL == 1) {
        (void)y;
        p[0] = uint32_t(__builtin_amdgcn_update_dpp(0, int(v[0]), 0x111, 0xF, 0xF, true));
    } else {
        p[0] = uint32_t(__builtin_amdgcn_update_dpp(0, int(v[0]), 0x111, 0xF, 0xF, true));
        const uint32_t t1 = uint32_t(__builtin_amdgcn_update_dpp(0, int(v[1]), 0x111, 0xF, 0xF, true));
        const uint32_t w0 = uint32_t(__builtin_amdgcn_update_dpp(0, int(v[0]), 0x121, 0xF, 0xF, true));
        p[1] = y == 0 ? w0 : t1;
    }
}

template <int RPL>
__device__ inline bool any_row(const uint32_t (&v)[RPL]) {
    uint32_t o = 0u;
#pragma unroll
    for (int h = 0; h < RPL; ++h) o |= v[h];
    return o != 0u;
}

// Count the votes of rule r's channel-list entries lo .. hi - 1 (packed r | i << 8 | j << 16 |
// plus << 24) into the KB-bit bit-sliced counters cnt of the lane's rows yr: a plus vote adds
// its cells, a minus vote adds the complement of its cells; nm counts the minus entries.  Four
// entries at a time: carry-save adders make the four one-bit planes a 3-bit number, then one
// ripple add.
template <int KB, int RPL>
__device__ inline void count_votes(uint32_t (&cnt)[RPL][KB], int &nm, const uint32_t *vl, int lo,
                                   int hi, const uint32_t *Mr, const int (&yr)[RPL],
                                   const bool (&rw)[RPL]) {
    for (int ev = lo; ev < hi; ev += 4) {
        uint32_t v[4];
        bool live[4], minus[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = vl[min(ev + u, hi - 1)];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            live[u] = ev + u < hi;
            minus[u] = live[u] && !((v[u] >> 24) & 1u);
            nm += minus[u] ? 1 : 0;
        }
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
            uint32_t x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint32_t t =
                    rw[h] ? Mr[yr[h] - int((v[u] >> 8) & 255u)] << ((v[u] >> 16) & 255u) : 0u;
                x[u] = !live[u] ? 0u : minus[u] ? ~t : t;
            }
            const uint32_t a = x[0] ^ x[1], s1 = a ^ x[2];
            const uint32_t c1 = (x[0] & x[1]) | (x[2] & a);            // weight 2
            const uint32_t s0 = s1 ^ x[3], c2 = s1 & x[3];             // weight 1, 2
            const uint32_t w2 = c1 ^ c2, w4 = c1 & c2;                 // weight 2, 4
            uint32_t *const q = cnt[h];
            uint32_t k = q[0] & s0;
            q[0] ^= s0;
            const uint32_t a1 = q[1] ^ w2;
            const uint32_t k1 = (q[1] & w2) | (k & a1);
            q[1] = a1 ^ k;
            const uint32_t a2 = q[2] ^ w4;
            k = (q[2] & w4) | (k1 & a2);
            q[2] = a2 ^ k1;
#pragma unroll
            for (int b = 3; b < KB; ++b) {
                const uint32_t kq = q[b] & k;
                q[b] ^= k;
                k = kq;
            }
        }
    }
}

// The exact write of channel c for the lane's rows (needed only where some cell of the group
// got votes of both signs): the votes on c of every rule in `fired` (the channel's vote list
// `vl`, ordered by rule; rule r's entries are vl[rsc[r] & 0xFFFF .. rsc[r] >> 16)) with the old
// value as a plus vote.  One counter takes old + #plus + (#minus entries - #minus votes), so a
// cell is set, old + #plus - #minus >= 1, where it reaches 1 + #minus entries.  A list holds
// at most 254 entries (eligibility: every entry is a distinct rule and pattern cell), so
// 8-bit counters never overflow; 4 bits do when the fired rules' entries are at most 14.
// With `moves` (the player plane) the four moves' votes, two entries each (-1 on the player's
// cell, +1 on the cell it moves to), are read from their match rows at once: the counter starts
// at old + their four plus votes + (4 - their four minus votes) and only the loaded rules'
// lists are walked.  (The four-wave kernels of groups of up to two rules, whose probe rows stay
// in registers, walk the moves too: the start's registers would spill the step's own.)
template <int RPL>
__device__ inline void exact_channel(const uint32_t (&old)[RPL], uint64_t fired, bool moves,
                                     const uint32_t *vl, const uint32_t *rsc, const uint32_t *M,
                                     int MS, int pad, const int (&yr)[RPL], const bool (&rw)[RPL],
                                     uint32_t (&out)[RPL]) {
    const uint64_t walk = moves ? fired & ~((1ull << kMoveRules) - 1ull) : fired;
    int total = moves ? 2 * kMoveRules : 0;
    for (uint64_t fr = walk; fr; fr &= fr - 1) {
        const uint32_t rs = rsc[__builtin_ctzll(fr)];
        total += int(rs >> 16) - int(rs & 0xFFFFu);
    }
    int nm = moves ? kMoveRules : 0;
    auto ge = [&](auto &cnt, auto kb) {           // cnt >= 1 + nm, bit-sliced
        constexpr int KB = decltype(kb)::value;
        const uint32_t T = uint32_t(1 + nm);
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
            uint32_t gt = 0u, eq = ~0u;
#pragma unroll
            for (int q = KB - 1; q >= 0; --q) {
                const uint32_t tb = ((T >> q) & 1u) ? ~0u : 0u;
                gt |= eq & cnt[h][q] & ~tb;
                eq &= ~(cnt[h][q] ^ tb);
            }
            out[h] = gt | eq;
        }
    };
    auto run = [&](auto kb) {
        constexpr int KB = decltype(kb)::value;
        uint32_t cnt[RPL][KB];
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
#pragma unroll
            for (int q = 0; q < KB; ++q) cnt[h][q] = 0u;
            const uint32_t o = rw[h] ? old[h] : 0u;
            if (moves) {
                // match rows of right, left, down, up (rules 0..3) at this row and the one above
                const uint32_t *m = M + pad + yr[h];
                const uint32_t m0 = m[0], m1 = m[MS], m2 = m[2 * MS], m3 = m[3 * MS];
                const uint32_t m2p = m[2 * MS - 1], m3p = m[3 * MS - 1];
                const uint32_t a1 = m0 << 1, b2 = m1 << 1;
                // plus: old, a1, m1, m2p, m3 -> p2 p1 p0
                const uint32_t s1 = o ^ a1 ^ m1, c1 = (o & a1) | (m1 & (o ^ a1));
                const uint32_t p0 = s1 ^ m2p ^ m3, c2 = (s1 & m2p) | (m3 & (s1 ^ m2p));
                const uint32_t p1 = c1 ^ c2, p2 = c1 & c2;
                // complements of the minus votes m0, b2, m2, m3p -> q2 q1 q0 (4 - their sum)
                const uint32_t s3 = m0 ^ b2 ^ m2, c3 = (m0 & b2) | (m2 & (m0 ^ b2));
                const uint32_t q0 = s3 ^ m3p, q1 = c3 ^ (s3 | m3p), q2 = ~(c3 | s3 | m3p);
                // p + q (at most 9)
                const uint32_t k0 = p0 & q0;
                const uint32_t k1 = (p1 & q1) | (k0 & (p1 ^ q1));
                const uint32_t k2 = (p2 & q2) | (k1 & (p2 ^ q2));
                cnt[h][0] = p0 ^ q0;
                cnt[h][1] = p1 ^ q1 ^ k0;
                cnt[h][2] = p2 ^ q2 ^ k1;
                cnt[h][3] = k2;
            } else {
                cnt[h][0] = o;
            }
        }
        for (uint64_t fr = walk; fr; fr &= fr - 1) {
            const int r = __builtin_ctzll(fr);
            const uint32_t rs = rsc[r];
            count_votes<KB, RPL>(cnt, nm, vl, int(rs & 0xFFFFu), int(rs >> 16),
                                 M + r * MS + pad, yr, rw);
        }
        ge(cnt, kb);
    };
    if (total <= 14) run(std::integral_constant<int, 4>{});
    else run(std::integral_constant<int, kCountBits>{});
}

// NR: rules a group holds (a bound on this launch's ceil(R / G)).
// RPL: map rows a lane holds: 2 on maps of 17 to 32 rows (lane y of a 16-lane group holds rows
// y and y + 16), else 1.
// NJ: columns a merged entry tests (3 when no pattern is wider, else 8).
// PROG_LDS: the rule program is copied to LDS.  A compile-time choice, so that the program's
// reads are LDS reads or global loads: a pointer that may be either makes every read a flat
// load, which the LDS reads' waits then wait for as well.
// SHORT: a launch of fewer than 16 steps (one step per observation), whose time is its set-up,
// a step or a few and the final store, each a chain of memory round trips: every load of the
// set-up is issued before its LDS writes (copy loops that wait for each load are one round
// trip per 64 words), the final store forms its addresses anew, and the kernel may take 256
// VGPRs, so nothing spills to scratch (at 128 a cold scratch reload on the path costs a round
// trip).  Longer launches keep four waves per SIMD and the per-row set-up, whose step loop
// measured faster (the set-up's code changes the loop's register assignment).
// WIDE: a batch of at most two waves per SIMD (program in LDS), which four-wave occupancy
// would not serve: the kernel may take 256 VGPRs, so nothing spills.
template <int Hq, int RPL, int NR, int NJ, bool PROG_LDS, bool SHORT, bool WIDE>
__global__ void __launch_bounds__(64, NR <= 8 ? ((SHORT || WIDE) ? 2 : 4) : 1) group_step(StepArgs a) {
    static_assert(RPL == 1 || Hq == 16, "two rows a lane in 16-lane groups");
    static_assert(!(SHORT && PROG_LDS), "short launches read the program from global memory");
    static_assert(!(WIDE && (SHORT || !PROG_LDS)), "wide kernels are long launches with the program in LDS");
    constexpr int G = 64 / Hq;
    constexpr int HR = Hq * RPL;              // map rows a group covers
    constexpr int kChunk = 4;                 // entries or votes of a rule read in one round
    extern __shared__ __align__(16) uint32_t lds[];
    const int lane = int(threadIdx.x), g = lane / Hq, y = lane % Hq;
    const uint64_t t_start = __builtin_amdgcn_s_memtime();
    const int b = a.order ? a.order[blockIdx.x] : int(blockIdx.x);
    const int H = a.H, W = a.W, C = a.C, C1 = C + 1, Rt = a.prog.rules_per_set;
    // pattern rows beyond a lane's row: plane rows y + i and match rows y - i, i <= PAD, are
    // read without a bounds test; rows of 4 words keep the probe table 16-byte aligned
    const int PAD = a.max_pat_h - 1;
    const int PR = group_plane_words(HR, a.max_pat_h), MS = PR;
    const int s = a.per_env ? b : 0;
    // the lane's rows; past the map (rw false) their plane rows stay zero and are read freely
    // (row yr + i < PR), their anchors are masked off and they are never written
    int yr[RPL];
    bool rw[RPL];
#pragma unroll
    for (int h = 0; h < RPL; ++h) {
        yr[h] = y + Hq * h;
        rw[h] = yr[h] < H;
    }
    const uint32_t wmask = low_mask(W);

    uint32_t *P = lds;                             // [C1][PR]
    uint32_t *M = P + C1 * PR;                     // [Rt][MS]
    uint32_t *PL = M + Rt * MS;                    // [C][HR]
    uint32_t *MI = PL + C * HR;                    // [C][HR]
    uint32_t *I0 = MI + C * HR;                    // [C][HR] initial rows
    uint32_t *PT = I0 + C * HR;                    // [Rt + 1][kProbeWords] probe table
    uint32_t *RS = PT + (Rt + 1) * kProbeWords;    // [C][Rt] rule ranges of channel lists
    uint32_t *RM = RS + C * Rt;                    // [C][2] rules with votes on each channel
    uint32_t *lprog = RM + 2 * C;                  // program copy (PROG_LDS)

    const uint32_t *ghdr = reinterpret_cast<const uint32_t *>(a.prog.hdr + size_t(s) * Rt);
    const uint32_t *gment = a.prog.gmatch + size_t(s) * a.prog.gmatch_stride;
    const uint32_t *gvent = a.prog.rvote + size_t(s) * a.prog.rvote_stride;
    const uint32_t *gvl = reinterpret_cast<const uint32_t *>(a.prog.votes + size_t(s) * C1);
    const uint32_t *gvote = a.prog.vote + size_t(s) * a.prog.vote_stride;
    const int hdr_words = Rt * kHdrWords;
    const uint32_t *hdrw = ghdr, *ment = gment, *vent = gvent, *vlw = gvl, *vote = gvote;
    if constexpr (PROG_LDS) {
        uint32_t *ph = lprog, *pm = ph + hdr_words, *pv = pm + a.prog.gmatch_stride;
        uint32_t *pl = pv + a.prog.rvote_stride, *pc = pl + 2 * C1;
        for (int w = lane; w < hdr_words; w += 64) ph[w] = ghdr[w];
        for (int w = lane; w < a.prog.gmatch_stride; w += 64) pm[w] = gment[w];
        for (int w = lane; w < a.prog.rvote_stride; w += 64) pv[w] = gvent[w];
        for (int w = lane; w < 2 * C1; w += 64) pl[w] = gvl[w];
        for (int w = lane; w < a.prog.vote_stride; w += 64) pc[w] = gvote[w];
        hdrw = ph;
        ment = pm;
        vent = pv;
        vlw = pl;
        vote = pc;
    }
    {
        const int words = C1 * PR + Rt * MS + 3 * C * HR;   // (PT and RS are copied)
        for (int w = lane; w < words; w += 64) lds[w] = 0u;
    }

    // the probe table and the rule ranges (built with the program: compile_group_tables)
    {
        const uint32_t *gt = a.prog.gtab + size_t(s) * a.prog.gtab_stride;
        if constexpr (SHORT) copy_to_lds(PT, gt, a.prog.gtab_stride, lane);
        else for (int w = lane; w < a.prog.gtab_stride; w += 64) PT[w] = gt[w];
    }
    const int nl = Rt - kMoveRules;               // loaded rules
    const int nr = (nl - g + G - 1) / G;          // this group's loaded rule count
    // (SHORT) lane l takes row l % H of channels l / H, l / H + 64 / H, ...
    const int rcs = 64 / H;
    if constexpr (SHORT) {
        const int rcl = lane / H, rrow = lane - rcl * H;
        auto load_rows = [&](const auto *st, const auto *in) {
            for (int c0 = rcl; c0 < C; c0 += 4 * rcs) {
                uint32_t sv[4], iv[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int c = c0 + u * rcs;
                    const size_t at = (size_t(c) * a.B + b) * H + rrow;
                    sv[u] = c < C ? uint32_t(st[at]) : 0u;
                    iv[u] = c < C ? uint32_t(in[at]) : 0u;
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int c = c0 + u * rcs;
                    if (c < C) {
                        P[c * PR + rrow] = sv[u];
                        I0[c * HR + rrow] = iv[u];
                    }
                }
            }
        };
        if (rcl < rcs) {
            if (a.row_bytes == 2)
                load_rows(static_cast<const uint16_t *>(a.state), static_cast<const uint16_t *>(a.init));
            else
                load_rows(static_cast<const uint32_t *>(a.state), static_cast<const uint32_t *>(a.init));
        }
    } else {
#pragma unroll
    for (int q = 0; q < kMaxChanPerGroup; ++q) {
        const int c = g + G * q;
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
            if (c < C && rw[h]) {
                const size_t at = (size_t(c) * a.B + b) * H + yr[h];
                P[c * PR + yr[h]] = a.row_bytes == 2
                                        ? uint32_t(static_cast<const uint16_t *>(a.state)[at])
                                        : static_cast<const uint32_t *>(a.state)[at];
                I0[c * HR + yr[h]] = a.row_bytes == 2
                                         ? uint32_t(static_cast<const uint16_t *>(a.init)[at])
                                         : static_cast<const uint32_t *>(a.init)[at];
            }
        }
    }
    }
    __syncthreads();   // (one wave: orders the set-up's LDS writes before the step's reads)
    int t_env = a.t[b];
    const uint64_t nbase = a.nctr[b];

    // entry e (merged per plane row) at this lane's row: OR-s into bad the anchors where a
    // tested column does not hold the wanted value (the row moved right by the column's
    // offset); a column's care and want bits sign-extended are all-ones masks
    auto miss = [&](uint32_t e, uint32_t (&bad)[RPL]) {
        uint32_t v[RPL];
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
            v[h] = P[int(e & uint32_t(kMaxEntryOffset)) + yr[h]];
            if constexpr (NJ > 3) v[h] >>= (e >> 9) & 24u;
        }
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const uint32_t want = uint32_t(int32_t(e << (7 - j)) >> 31);
            const uint32_t care = uint32_t(int32_t(e << (15 - j)) >> 31);
#pragma unroll
            for (int h = 0; h < RPL; ++h) bad[h] |= ((v[h] >> j) ^ want) & care;
        }
    };
    // the anchors m of the lane's rows that pass four entries more
    auto entries4 = [&](uint32_t e0, uint32_t e1, uint32_t e2, uint32_t e3, uint32_t (&m)[RPL]) {
        uint32_t bad[RPL];
#pragma unroll
        for (int h = 0; h < RPL; ++h) bad[h] = 0u;
        miss(e0, bad);
        miss(e1, bad);
        miss(e2, bad);
        miss(e3, bad);
#pragma unroll
        for (int h = 0; h < RPL; ++h) m[h] &= ~bad[h];
    };

    uint32_t ablk = 0u;     // lane l: action of step k0 + l of the current block of 64
    float rbuf = 0.f;       // lane l: reward of step k0 + l
    uint32_t dbuf = 0u;     // lane l: done flag of step k0 + l
    uint32_t *const F = P + C * PR;
    uint32_t *const P2w = P + kChPlayer * PR;
    const uint32_t *const P2 = P2w;

    const uint32_t cm1 = low_mask(W - 1);         // anchors of a 1 x 2 pattern
    uint32_t vrow2[RPL];                          // rows of a 2 x 1 pattern's anchors
#pragma unroll
    for (int h = 0; h < RPL; ++h) vrow2[h] = (yr[h] + 2 <= H) ? wmask : 0u;
    const int pown = kChPlayer % G;               // the group that writes the player plane
    // the player and wall rows of the lane (every group holds them): the next step's follow
    // from the moves' votes in registers unless a loaded rule voted on either plane or the
    // episode ended; then they are read again
    uint32_t Pyr[RPL], Wyr[RPL];
#pragma unroll
    for (int h = 0; h < RPL; ++h) {
        Pyr[h] = rw[h] ? P2[yr[h]] : 0u;
        Wyr[h] = rw[h] ? P[kChWall * PR + yr[h]] : 0u;
    }
    // the probe rows of the group's rules: read once when the group has at most two rules,
    // else every step (registers would spill)
    uint4 pe[NR];
    uint32_t pv[NR];
    uint4 pe2[NR];                                // entries 4 .. 7 (NR <= 2)
    uint32_t pm[NR];                              // match offset | count << 16 (NR <= 2)
    if constexpr (NR <= 2) {
#pragma unroll
        for (int kr = 0; kr < NR; ++kr) {
            const int r = kr < nr ? kMoveRules + g + G * kr : kMoveRules;
            pe[kr] = *reinterpret_cast<const uint4 *>(PT + r * kProbeWords);
            pv[kr] = PT[r * kProbeWords + 4];
            pe2[kr] = *reinterpret_cast<const uint4 *>(PT + r * kProbeWords + 8);
            pm[kr] = kr < nr ? PT[r * kProbeWords + 5] : 0u;
        }
    }
    for (int k = 0; k < a.k; ++k) {
        const int kb = k & 63;
        if (kb == 0) ablk = (k + lane < a.k) ? uint32_t(a.actions[size_t(k + lane) * a.B + b]) : 0u;
        const int act = __builtin_amdgcn_readlane(int(ablk), kb);
        // the lane's rows of the player and wall planes (0 past the map; kept in registers
        // from step to step), and the probe table rows of the group's rules
        uint32_t Py[RPL], Wy[RPL];
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
            Py[h] = Pyr[h];
            Wy[h] = Wyr[h];
        }
        if constexpr (NR > 2) {                   // (up to two rules: held for the launch)
#pragma unroll
            for (int kr = 0; kr < NR; ++kr) {
                const int r = kr < nr ? kMoveRules + g + G * kr : kMoveRules;
                pe[kr] = *reinterpret_cast<const uint4 *>(PT + r * kProbeWords);
                pv[kr] = PT[r * kProbeWords + 4];
            }
        }
        // the rows next to them and the force row
        uint32_t Pn[RPL], Wn[RPL], Pp[RPL], Fy[RPL], Fn[RPL];
        next_rows<Hq, RPL>(Py, Pn, lane, y);
        next_rows<Hq, RPL>(Wy, Wn, lane, y);
        prev_rows<Hq, RPL>(Py, Pp, lane, y);
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
            Fy[h] = act == 1 ? Pn[h] : act == 3 ? Pp[h] : act == 2 ? ((Py[h] << 1) & wmask)
                  : act == 4 ? (Py[h] >> 1) : 0u;
            if (g == 0 && rw[h]) F[yr[h]] = Fy[h];
        }
        next_rows<Hq, RPL>(Fy, Fn, lane, y);
        // the four moves (rules 0..3: right, left, down, up) and their votes on the player
        // plane; group 0 stores their match rows for an exact recount
        uint32_t m0[RPL], m1[RPL], m2[RPL], m3[RPL], m2p[RPL], m3p[RPL];
        uint32_t mplus[RPL], mminus[RPL], pnew[RPL];
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
            m0[h] = Py[h] & (Fy[h] >> 1) & ~(Wy[h] >> 1) & cm1;
            m1[h] = Fy[h] & ~Wy[h] & (Py[h] >> 1) & cm1;
            m2[h] = Py[h] & Fn[h] & ~Wn[h] & vrow2[h];
            m3[h] = Fy[h] & ~Wy[h] & Pn[h] & vrow2[h];
        }
        prev_rows<Hq, RPL>(m2, m2p, lane, y);
        prev_rows<Hq, RPL>(m3, m3p, lane, y);
        uint32_t both = 0u;
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
            mplus[h] = (m0[h] << 1) | m1[h] | m2p[h] | m3[h];
            mminus[h] = m0[h] | (m1[h] << 1) | m2[h] | m3p[h];
            // the player rows after the moves' votes alone: one sign OR-ed, or, where some cell
            // got votes of both signs (players moving into cells other players leave), counted
            // exactly in registers: old + #plus > #minus over the four plus and four minus terms
            pnew[h] = (Py[h] | mplus[h]) & ~mminus[h];
            both |= mplus[h] & mminus[h];
        }
        if (__builtin_amdgcn_ballot_w64(both != 0u)) {
#pragma unroll
            for (int h = 0; h < RPL; ++h) {
                const uint32_t a1 = m0[h] << 1, b2 = m1[h] << 1, o = Py[h];
                // plus: old, a1, m1, m2p, m3 -> p2 p1 p0 (at most 5)
                const uint32_t s1 = o ^ a1 ^ m1[h], c1 = (o & a1) | (m1[h] & (o ^ a1));
                const uint32_t p0 = s1 ^ m2p[h] ^ m3[h], c2 = (s1 & m2p[h]) | (m3[h] & (s1 ^ m2p[h]));
                const uint32_t p1 = c1 ^ c2, p2 = c1 & c2;
                // minus: m0, b2, m2, m3p -> n2 n1 n0 (at most 4)
                const uint32_t s3 = m0[h] ^ b2 ^ m2[h], c3 = (m0[h] & b2) | (m2[h] & (m0[h] ^ b2));
                const uint32_t n0 = s3 ^ m3p[h], c4 = s3 & m3p[h];
                const uint32_t n1 = c3 ^ c4, n2 = c3 & c4;
                pnew[h] = (p2 & ~n2) | (~(p2 ^ n2) & ((p1 & ~n1) | (~(p1 ^ n1) & p0 & ~n0)));
            }
        }
        if (g == 0) {
#pragma unroll
            for (int h = 0; h < RPL; ++h) {
                M[0 * MS + PAD + yr[h]] = m0[h];
                M[1 * MS + PAD + yr[h]] = m1[h];
                M[2 * MS + PAD + yr[h]] = m2[h];
                M[3 * MS + PAD + yr[h]] = m3[h];
            }
        }
        uint64_t fired = (__builtin_amdgcn_ballot_w64(any_row<RPL>(m0)) ? 1ull : 0ull) |
                         (__builtin_amdgcn_ballot_w64(any_row<RPL>(m1)) ? 2ull : 0ull) |
                         (__builtin_amdgcn_ballot_w64(any_row<RPL>(m2)) ? 4ull : 0ull) |
                         (__builtin_amdgcn_ballot_w64(any_row<RPL>(m3)) ? 8ull : 0ull);

        // probe: every loaded rule of the group with its first four entries, all reads at once
        // (no branch between the rules); the results go to the rules' match rows, and a
        // wave-uniform mask of the rule indices kr whose probe passed in some group
        uint32_t mk[NR][RPL];
#pragma unroll
        for (int kr = 0; kr < NR; ++kr) {
#pragma unroll
            for (int h = 0; h < RPL; ++h)
                mk[kr][h] = (kr < nr && yr[h] < int(pv[kr] >> 8)) ? ~0u >> (pv[kr] & 255u) : 0u;
            entries4(pe[kr].x, pe[kr].y, pe[kr].z, pe[kr].w, mk[kr]);
        }
        uint32_t cand = 0u;
#pragma unroll
        for (int kr = 0; kr < NR; ++kr) {
            if (kr < nr) {
#pragma unroll
                for (int h = 0; h < RPL; ++h)
                    M[(kMoveRules + g + G * kr) * MS + PAD + yr[h]] = mk[kr][h];
            }
            cand |= __builtin_amdgcn_ballot_w64(any_row<RPL>(mk[kr])) ? 1u << kr : 0u;
        }

        // candidates: the rest of their input entries four at a time.  With up to four rules per
        // group, in rounds in which every candidate of every group takes its next four (a lane
        // only while it still holds an anchor of the rule; otherwise the pass entry, which
        // tests nothing; a rule slot no group still needs is skipped); with more, one rule after another, the next four entries
        // read while the current ones' plane rows are (rounds would issue every rule's reads
        // while most rules are done, and four waves share each CU's LDS there).  A rule is done
        // when its entries run out or its lanes have no anchor left.
        int rsum = 0;
        uint32_t voted = 0u;                      // bit c: a loaded rule voted on channel c
        if (cand) {
            uint32_t meta[NR];                    // match offset | entry count << 16
#pragma unroll
            for (int kr = 0; kr < NR; ++kr) {
                const int r = kr < nr ? kMoveRules + g + G * kr : kMoveRules;
                if constexpr (NR <= 2) meta[kr] = pm[kr];
                else meta[kr] = kr < nr ? PT[r * kProbeWords + 5] : 0u;
            }
            if constexpr (NR <= 4) {
                for (int e = kProbeEntries;; e += 4) {
                    // the rule slots still live in some group (the others are skipped)
                    uint32_t lk = 0u;
#pragma unroll
                    for (int kr = 0; kr < NR; ++kr)
                        lk |= __builtin_amdgcn_ballot_w64(any_row<RPL>(mk[kr]) && e < int(meta[kr] >> 16))
                                  ? 1u << kr : 0u;
                    if (!lk) break;
                    uint32_t x[NR][4];
#pragma unroll
                    for (int kr = 0; kr < NR; ++kr) {
                        if (!((lk >> kr) & 1u)) continue;
                        const int off = int(meta[kr] & 0xFFFFu), cnt = int(meta[kr] >> 16);
                        const bool live = any_row<RPL>(mk[kr]) && e < cnt;
                        if (NR <= 2 && e == kProbeEntries) {   // entries 4 .. 7: in registers
                            const uint4 q = pe2[kr];
                            x[kr][0] = live ? q.x : kPassEntry;
                            x[kr][1] = live ? q.y : kPassEntry;
                            x[kr][2] = live ? q.z : kPassEntry;
                            x[kr][3] = live ? q.w : kPassEntry;
                            continue;
                        }
                        if (NR > 2 && e == kProbeEntries) {    // entries 4 .. 7: the probe row's
                            const int r = kr < nr ? kMoveRules + g + G * kr : kMoveRules;
#pragma unroll
                            for (int u = 0; u < 4; ++u)
                                x[kr][u] = live ? PT[r * kProbeWords + 8 + u] : kPassEntry;
                            continue;
                        }
#pragma unroll
                        for (int u = 0; u < 4; ++u) {
                            // past the last entry the last one again (AND is idempotent)
                            const uint32_t w = ment[live ? off + min(e + u, cnt - 1) : 0];
                            x[kr][u] = live ? w : kPassEntry;
                        }
                    }
#pragma unroll
                    for (int kr = 0; kr < NR; ++kr)
                        if ((lk >> kr) & 1u) entries4(x[kr][0], x[kr][1], x[kr][2], x[kr][3], mk[kr]);
                }
            } else {
#pragma unroll
                for (int kr = 0; kr < NR; ++kr) {
                    if (!((cand >> kr) & 1u)) continue;
                    uint32_t m[RPL];
#pragma unroll
                    for (int h = 0; h < RPL; ++h) m[h] = mk[kr][h];
                    if (!(kr < nr && group_any<Hq>(any_row<RPL>(m), lane))) continue;
                    const uint32_t *en = ment + int(meta[kr] & 0xFFFFu);
                    const int cnt = int(meta[kr] >> 16), last = cnt - 1;
                    int e = kProbeEntries;
                    uint32_t x[4] = {kPassEntry, kPassEntry, kPassEntry, kPassEntry};
                    if (e < cnt) {                // (reads stay inside the rule's entries)
#pragma unroll
                        for (int u = 0; u < 4; ++u) x[u] = en[min(e + u, last)];
                    }
                    while (e < cnt && group_any<Hq>(any_row<RPL>(m), lane)) {
                        uint32_t cur[4];
#pragma unroll
                        for (int u = 0; u < 4; ++u) cur[u] = x[u];
                        e += 4;
                        if (e < cnt) {
#pragma unroll
                            for (int u = 0; u < 4; ++u) x[u] = en[min(e + u, last)];
                        }
                        entries4(cur[0], cur[1], cur[2], cur[3], m);
                    }
#pragma unroll
                    for (int h = 0; h < RPL; ++h) mk[kr][h] = m[h];
                }
            }
            // the rules that fired in some group: match row, reward and votes
            uint32_t fl = 0u;
#pragma unroll
            for (int kr = 0; kr < NR; ++kr)
                fl |= __builtin_amdgcn_ballot_w64(any_row<RPL>(mk[kr])) ? 1u << kr : 0u;
            for (; fl; fl &= fl - 1u) {
                const int kr = __builtin_ctz(fl);
                const int r = kMoveRules + g + G * kr;
                uint32_t m[RPL];                  // mk[kr] (kr is wave-uniform)
#pragma unroll
                for (int h = 0; h < RPL; ++h) m[h] = 0u;
#pragma unroll
                for (int kk = 0; kk < NR; ++kk) {
#pragma unroll
                    for (int h = 0; h < RPL; ++h) m[h] = kk == kr ? mk[kk][h] : m[h];
                }
                if (kr < nr && group_any<Hq>(any_row<RPL>(m), lane)) {
                    const uint32_t *hw = hdrw + r * kHdrWords;
                    int cells = 0;
#pragma unroll
                    for (int h = 0; h < RPL; ++h) {
                        M[r * MS + PAD + yr[h]] = m[h];
                        cells += __popc(m[h]);
                    }
                    fired |= 1ull << r;
                    // the vote list's place and the voted channels: with the program in global
                    // memory from the probe row (LDS), a memory round trip less before the votes
                    int voff, vcnt;
                    if constexpr (PROG_LDS) {
                        voted |= hw[7];
                        rsum += int(hw[2]) * cells;
                        voff = int(hw[5]);
                        vcnt = int(hw[6]);
                    } else {
                        const uint32_t pvw = PT[r * kProbeWords + 6];
                        voted |= PT[r * kProbeWords + 7];
                        rsum += int(hw[2]) * cells;
                        voff = int(pvw & 0xFFFFu);
                        vcnt = int(pvw >> 16);
                    }
                    // votes kChunk at a time, the next chunk read with the current one's match
                    // rows (a repeated last vote ORs the same bits again)
                    const uint32_t *ve = vent + voff;
                    const int vlast = vcnt - 1;
                    uint32_t v[kChunk];
                    if (vcnt > 0) {
#pragma unroll
                        for (int u = 0; u < kChunk; ++u) v[u] = ve[min(u, vlast)];
                    }
                    for (int ev = 0; ev < vcnt; ev += kChunk) {
                        uint32_t cv[kChunk], tv[kChunk][RPL];
#pragma unroll
                        for (int u = 0; u < kChunk; ++u) cv[u] = v[u];
                        if (ev + kChunk < vcnt) {
#pragma unroll
                            for (int u = 0; u < kChunk; ++u) v[u] = ve[min(ev + kChunk + u, vlast)];
                        }
#pragma unroll
                        for (int u = 0; u < kChunk; ++u) {
#pragma unroll
                            for (int h = 0; h < RPL; ++h)
                                tv[u][h] = M[r * MS + PAD + yr[h] - int((cv[u] >> 8) & 255u)]
                                           << ((cv[u] >> 16) & 255u);
                        }
#pragma unroll
                        for (int u = 0; u < kChunk; ++u) {
#pragma unroll
                            for (int h = 0; h < RPL; ++h)
                                if (rw[h] && tv[u][h])
                                    atomicOr(((cv[u] >> 24) & 1u ? PL : MI) + int(cv[u] & 255u) * HR + yr[h],
                                             tv[u][h]);
                        }
                    }
                }
            }
        }
        // every rule that fired anywhere in the wave and every channel a loaded rule voted on
        // (the groups' masks OR-ed)
        uint64_t fired_all = fired & 15ull;       // (the moves' bits are the same in every lane)
        uint32_t lvoted = 0u;                     // channels the loaded rules voted on
        if (__builtin_amdgcn_ballot_w64((fired >> kMoveRules) != 0ull)) {
#pragma unroll
            for (int gg = 0; gg < G; ++gg) {
                const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(fired)), gg * Hq));
                const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(fired >> 32)), gg * Hq));
                fired_all |= uint64_t(lo) | (uint64_t(hi) << 32);
                lvoted |= uint32_t(__builtin_amdgcn_readlane(int(voted), gg * Hq));
            }
        }
        const uint32_t voted_all = lvoted | ((fired_all & 15ull) ? 1u << kChPlayer : 0u);

        // new rows of the channels that received votes: group g rewrites channels g, g + G, ...
        // (the moves' votes on the player plane are in registers, the loaded rules' in LDS)
        bool pl_any = false;                      // a player bit after the write
#pragma unroll
        for (int h = 0; h < RPL; ++h) pl_any |= g == pown && rw[h] && Py[h] != 0u;
        if (voted_all == (1u << kChPlayer) && lvoted == 0u) {
            // only the moves voted (most steps): the player plane, from registers
            if (g == pown) {
                pl_any = false;
#pragma unroll
                for (int h = 0; h < RPL; ++h) {
                    if (rw[h]) P2w[yr[h]] = pnew[h];
                    pl_any |= rw[h] && pnew[h] != 0u;
                }
            }
        } else if (voted_all) {
#pragma unroll 1
            for (int c = g; c < C; c += G) {
                if (!((voted_all >> c) & 1u)) continue;
                const bool lv = (lvoted >> c) & 1u;
                uint32_t old[RPL], pl[RPL], mi[RPL], nw[RPL], mixed = 0u;
#pragma unroll
                for (int h = 0; h < RPL; ++h) {
                    old[h] = c == kChPlayer ? Py[h] : P[c * PR + yr[h]];
                    pl[h] = lv ? PL[c * HR + yr[h]] : 0u;
                    mi[h] = lv ? MI[c * HR + yr[h]] : 0u;
                    if (c == kChPlayer) {
                        pl[h] |= mplus[h];
                        mi[h] |= mminus[h];
                    }
                    nw[h] = (old[h] | pl[h]) & ~mi[h];
                    mixed |= pl[h] & mi[h];
                }
                if (c == kChPlayer && !lv) {
#pragma unroll
                    for (int h = 0; h < RPL; ++h) nw[h] = pnew[h];   // only the moves voted on it
                } else if (group_any<Hq>(mixed != 0u, lane)) {
                    exact_channel<RPL>(old, fired_all & (uint64_t(RM[2 * c]) | uint64_t(RM[2 * c + 1]) << 32),
                                       (NR > 2 || SHORT || WIDE) && c == kChPlayer, vote + int(vlw[2 * c]),
                                       RS + c * Rt, M, MS, PAD, yr, rw, nw);
                }
                if (c == kChPlayer) pl_any = false;
#pragma unroll
                for (int h = 0; h < RPL; ++h) {
                    if (rw[h]) P[c * PR + yr[h]] = nw[h];
                    if (c == kChPlayer) pl_any |= rw[h] && nw[h] != 0u;
                    if (lv) {
                        PL[c * HR + yr[h]] = 0u;
                        MI[c * HR + yr[h]] = 0u;
                    }
                }
            }
        }

        // reward: the lanes' sums over the wave
        if (__builtin_amdgcn_ballot_w64(rsum != 0)) {
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) rsum += __shfl_xor(rsum, off);
        }
        // episode end: a player bit left anywhere (the writing group's lanes hold the rows)
        const bool anyp = __builtin_amdgcn_ballot_w64(pl_any) != 0ull;
        t_env += 1;
        const bool d = !anyp || (a.L > 0 && t_env == a.L);
        if (d) {                                  // back to the initial rows
            t_env = 0;
#pragma unroll
            for (int h = 0; h < RPL; ++h) {
                if (rw[h]) {
#pragma unroll 1
                    for (int c = g; c < C; c += G) P[c * PR + yr[h]] = I0[c * HR + yr[h]];
                }
            }
        }
        if (d || ((lvoted >> kChPlayer) & 1u) || ((lvoted >> kChWall) & 1u)) {
#pragma unroll
            for (int h = 0; h < RPL; ++h) {
                Pyr[h] = rw[h] ? P2[yr[h]] : 0u;
                Wyr[h] = rw[h] ? P[kChWall * PR + yr[h]] : 0u;
            }
        } else {
#pragma unroll
            for (int h = 0; h < RPL; ++h) Pyr[h] = pnew[h];
        }
        if (lane == kb) {
            rbuf = float(rsum);
            dbuf = d ? 1u : 0u;
        }
        if (kb == 63 || k == a.k - 1) {
            const int k0 = k - kb;
            if (lane <= kb) {
                a.rewards[size_t(k0 + lane) * a.B + b] = rbuf;
                a.done[size_t(k0 + lane) * a.B + b] = uint8_t(dbuf);
            }
        }
    }

    if constexpr (SHORT) {
        // the rows back as they were read, the lane's channel and row formed again from an
        // opaque copy of its index (kept from the set-up they were spilled through the launch)
        int le = lane;
        asm volatile("" : "+v"(le));
        const int wcl = le / H, wrow = le - wcl * H;
        if (wcl < rcs) {
#pragma unroll 4
            for (int c = wcl; c < C; c += rcs) {
                const size_t at = (size_t(c) * a.B + b) * H + wrow;
                if (a.row_bytes == 2) static_cast<uint16_t *>(a.state)[at] = uint16_t(P[c * PR + wrow]);
                else static_cast<uint32_t *>(a.state)[at] = P[c * PR + wrow];
            }
        }
    } else {
#pragma unroll
    for (int q = 0; q < kMaxChanPerGroup; ++q) {
        const int c = g + G * q;
#pragma unroll
        for (int h = 0; h < RPL; ++h) {
            if (c < C && rw[h]) {
                const size_t at = (size_t(c) * a.B + b) * H + yr[h];
                if (a.row_bytes == 2) static_cast<uint16_t *>(a.state)[at] = uint16_t(P[c * PR + yr[h]]);
                else static_cast<uint32_t *>(a.state)[at] = P[c * PR + yr[h]];
            }
        }
    }
    }
    if (lane == 0) {
        a.t[b] = t_env;
        a.nctr[b] = nbase + uint64_t(a.k);
        if (a.cost) {
            const uint64_t c = (__builtin_amdgcn_s_memtime() - t_start) >> 8;
            a.cost[b] = uint32_t(c < 0xFFFFFFFFull ? c : 0xFFFFFFFFull);
        }
    }
}

}  // namespace

// Map rows a lane group covers: its 16 lanes hold one row each, or two on maps of 17 to 32 rows.
static int group_rows(int H) { return H <= 16 ? 16 : 32; }

size_t group_lds_bytes(int H, int C, int rules_per_set, int max_pat_h) {
    const int HR = group_rows(H), PR = group_plane_words(HR, max_pat_h);
    return sizeof(uint32_t) * (size_t(C + 1) * PR + size_t(rules_per_set) * PR +
                               size_t(3) * C * HR + size_t(rules_per_set + 1) * kProbeWords +
                               size_t(C) * (rules_per_set + 2));
}

bool group_eligible(int H, int W, int C, int rules_per_set, int max_pat_h, int max_pat_w) {
    if (H > 32 || W > 32) return false;
    // every vote a cell-channel gets comes from a distinct (rule, pattern cell): the 8-bit
    // counts of the exact write hold them (plus the old value) when there are at most 255
    if (long(rules_per_set) * max_pat_h * max_pat_w > 254) return false;
    constexpr int G = 4;                          // lane groups a wave holds
    // (merged entries address rows of the stored and force planes in 12 bits)
    return rules_per_set <= kMaxRulesPerGroup * G && rules_per_set <= 64 &&
           C <= kMaxChanPerGroup * G &&
           (C + 1) * group_plane_words(group_rows(H), max_pat_h) <= kMaxEntryOffset + 1 &&
           group_lds_bytes(H, C, rules_per_set, max_pat_h) <= size_t(kLdsBudget);
}

// A rule's input entries (c | i << 8 | j << 16 | want << 24, rarest first) merged per plane
// row and block of 8 columns, in the order of each row's first entry.
static std::vector<uint32_t> merge_entries(const uint32_t *ent, int cnt, int PR) {
    std::vector<uint32_t> key, out;               // key: c | i << 8 | jb << 16
    for (int e = 0; e < cnt; ++e) {
        const uint32_t c = ent[e] & 255u, i = (ent[e] >> 8) & 255u, j = (ent[e] >> 16) & 255u;
        const uint32_t k = c | (i << 8) | ((j >> 3) << 16), bit = 1u << (j & 7u);
        size_t q = 0;
        while (q < key.size() && key[q] != k) ++q;
        if (q == key.size()) {                    // no column tested yet
            key.push_back(k);
            out.push_back((c * uint32_t(PR) + i) | ((j >> 3) << 12));
        }
        out[q] |= bit << 16;                      // column tested
        if ((ent[e] >> 24) & 1u) out[q] |= bit << 24;   // must be 1
    }
    return out;
}

void compile_group_tables(const GenericProgram &p, int H, int W, int C, int max_pat_h,
                          std::vector<uint32_t> &tab, int &stride, std::vector<uint32_t> &gm,
                          int &gm_stride) {
    const int Rt = p.rules_per_set, C1 = C + 1;
    const int PR = group_plane_words(group_rows(H), max_pat_h);
    stride = (Rt + 1) * kProbeWords + C * Rt + 2 * C;
    tab.assign(size_t(p.sets) * stride, 0u);
    std::vector<std::vector<uint32_t>> merged(p.sets);
    gm_stride = 1;
    for (int s = 0; s < p.sets; ++s) {
        uint32_t *pt = tab.data() + size_t(s) * stride, *rs = pt + (Rt + 1) * kProbeWords;
        // probe rows of the loaded rules: the first four merged entries (a missing one always
        // passes) and the anchors, columns 0 .. W - m (~0 >> (32 - (W - m + 1))) of rows
        // 0 .. H - n
        for (int r = kMoveRules; r < Rt; ++r) {
            const RuleHdr &h = p.hdr[size_t(s) * Rt + r];
            const std::vector<uint32_t> ent = merge_entries(
                p.match.data() + size_t(s) * p.match_stride + h.match_off, h.match_cnt, PR);
            const int off = int(merged[s].size()), cnt = int(ent.size());
            merged[s].insert(merged[s].end(), ent.begin(), ent.end());
            uint32_t *row = pt + r * kProbeWords;
            for (int e = 0; e < kProbeEntries; ++e) row[e] = e < cnt ? ent[e] : kPassEntry;
            const int cols = W - h.m + 1, rows = H - h.n + 1;
            row[4] = (cols >= 1 && rows >= 1) ? uint32_t(32 - cols) | (uint32_t(rows) << 8) : 0u;
            row[5] = uint32_t(off) | (uint32_t(cnt) << 16);
            // the rule-major votes (a set holds at most 64 rules of at most 254 votes, so the
            // offset and count fit 16 bits each) and the channels they are on
            row[6] = uint32_t(h.vote_off) | (uint32_t(h.vote_cnt) << 16);
            row[7] = uint32_t(h.pad);
            // entries 4 .. 7 (past the last, the last again; none: the pass entry)
            for (int e = 0; e < 4; ++e)
                row[8 + e] = cnt > kProbeEntries ? ent[std::min(kProbeEntries + e, cnt - 1)]
                                                 : kPassEntry;
        }
        gm_stride = std::max(gm_stride, int(merged[s].size()));
        // rule ranges of the channel vote lists (each ordered by rule): first | end << 16
        for (int c = 0; c < C; ++c) {
            const VoteList &vl = p.votes[size_t(s) * C1 + c];
            const uint32_t *v = p.vote.data() + size_t(s) * p.vote_stride + vl.off;
            for (int k = 0; k < vl.cnt; ++k) {
                const int r = int(v[k] & 255u);
                uint32_t &w = rs[c * Rt + r];
                if (k == 0 || int(v[k - 1] & 255u) != r) w |= uint32_t(k);
                if (k == vl.cnt - 1 || int(v[k + 1] & 255u) != r) w |= uint32_t(k + 1) << 16;
                // the rules with votes on the channel, a 64-bit mask (an exact write visits
                // only the fired ones among them)
                rs[C * Rt + 2 * c + (r >> 5)] |= 1u << (r & 31);
            }
        }
    }
    gm.assign(size_t(p.sets) * gm_stride, kPassEntry);
    for (int s = 0; s < p.sets; ++s)
        std::copy(merged[s].begin(), merged[s].end(), gm.begin() + size_t(s) * gm_stride);
}

namespace {
template <int RPL, int NJ, bool PROG_LDS, bool SHORT, bool WIDE>
void launch_nr(const StepArgs &a, size_t lds, hipStream_t s) {
    constexpr int G = 4;
    const int nrmax = (a.prog.rules_per_set - kMoveRules + G - 1) / G;
    const dim3 grid(a.B), block(64);
    if (nrmax <= 2) hipLaunchKernelGGL((group_step<16, RPL, 2, NJ, PROG_LDS, SHORT, WIDE>), grid, block, lds, s, a);
    else if (nrmax <= 4) hipLaunchKernelGGL((group_step<16, RPL, 4, NJ, PROG_LDS, SHORT, WIDE>), grid, block, lds, s, a);
    else if (nrmax <= 8) hipLaunchKernelGGL((group_step<16, RPL, 8, NJ, PROG_LDS, SHORT, WIDE>), grid, block, lds, s, a);
    else if (nrmax <= 12) hipLaunchKernelGGL((group_step<16, RPL, 12, NJ, PROG_LDS, SHORT, WIDE>), grid, block, lds, s, a);
    else hipLaunchKernelGGL((group_step<16, RPL, 16, NJ, PROG_LDS, SHORT, WIDE>), grid, block, lds, s, a);
}
template <int RPL, int NJ>
void launch_rpl(const StepArgs &a, size_t lds, bool prog_lds, bool wide, hipStream_t s) {
    if (prog_lds && wide) launch_nr<RPL, NJ, true, false, true>(a, lds, s);
    else if (prog_lds) launch_nr<RPL, NJ, true, false, false>(a, lds, s);
    else if (a.k < kShortLaunch) launch_nr<RPL, NJ, false, true, false>(a, lds, s);
    else launch_nr<RPL, NJ, false, false, false>(a, lds, s);
}

// SIMDs of the current device (4 per compute unit), looked up once per device.
int device_simds() {
    static int simds[64] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1024;
    if (!simds[dev]) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
            return 1024;
        simds[dev] = 4 * cus;
    }
    return simds[dev];
}
}  // namespace

hipError_t launch_group_step(const StepArgs &a, hipStream_t s) {
    const size_t base = group_lds_bytes(a.H, a.C, a.prog.rules_per_set, a.max_pat_h);
    const size_t prog = sizeof(uint32_t) * (size_t(a.prog.rules_per_set) * kHdrWords +
                                            a.prog.gmatch_stride + a.prog.rvote_stride +
                                            2 * (a.C + 1) + a.prog.vote_stride);
    // the program goes to LDS for launches of 16 steps or more, when it fits and leaves room
    // for as many waves per CU (160 KiB of LDS) as the batch can use, up to 16 (4 per SIMD)
    const size_t need = size_t(std::min(16, (a.B + 255) / 256));
    const size_t budget = std::min(size_t(kLdsBudget), size_t(160) * 1024 / need);
    const bool prog_lds = a.k >= kShortLaunch && base + prog <= budget;
    const size_t lds = base + (prog_lds ? prog : 0);
    const bool narrow = a.max_pat_w <= 3;
    // at most two waves per SIMD: the 256-VGPR kernels
    const bool wide = a.B <= 2 * device_simds();
    if (group_rows(a.H) == 16) {
        if (narrow) launch_rpl<1, 3>(a, lds, prog_lds, wide, s);
        else launch_rpl<1, 8>(a, lds, prog_lds, wide, s);
    } else {
        if (narrow) launch_rpl<2, 3>(a, lds, prog_lds, wide, s);
        else launch_rpl<2, 8>(a, lds, prog_lds, wide, s);
    }
    return hipGetLastError();
}

}  // namespace av
