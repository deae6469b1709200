// wave engine: one environment per workgroup, its rules split over row groups.
//
// A workgroup holds one environment.  Its threads form G groups of Hq lanes (Hq = 16, 32 or
// 64 rows, the map height rounded up; G from 4 up to 1024 / Hq threads for 32-bit rows, 512 /
// Hq for 64-bit rows, the most for which the whole batch fits the device's wave slots at
// once, and no more than the rules need); lane y of every group owns map row y.  Group g evaluates rules g, g+G, g+2G, ... so G rules are matched at once, and
// with one environment per workgroup the environment's own rules need no per-lane selection:
// every lane of a group reads the same rule entry.  The rule program (headers, input
// entries rarest first, rule-major votes) is copied into LDS once per launch when it fits.
//
// LDS:
//   planes  [C+1][H+16] rows: the map and the force plane; 16 zero rows below the map let
//           a lane read row y+i of any pattern without a bounds test
//   match   [R+4][16+64] rows: match planes of the rules that fired (for exact counts)
//   plus, minus [C+1][64] rows: per plane, OR of the +1 and of the -1 votes
//   fired   [R+4] flags, reward accumulator, program copy
// Rows are 32-bit words for W <= 32, 64-bit for W <= 64; bit x = column x.
//
// Per step (paper Sec. 2.1, Sec. 2.1.1, Sec. 2.2.1), for one batch of all rules (parallel
// mode) or for one rule after another (sequential mode):
//   force   F[y] = the player row moved one cell toward the action;
//   match   per rule, AND over its specified entries of plane row y+i shifted right by j
//           (complemented for must-be-0), within the valid-anchor mask; a group leaves the
//           rule as soon as none of its lanes has a surviving anchor;
//   votes   right after a rule fired, each nonzero K_O = O - I entry takes the match row
//           y-i from the group's lane y-i (ds_bpermute), shifts it by j and ORs it into the
//           plus or minus row of its channel (LDS atomic OR);
//   write   new = (old | plus) & ~minus where no cell got both signs; a channel whose rows
//           have mixed cells is recounted exactly with bit-sliced counters of its plus and
//           minus votes: new = (old + #plus > #minus) = (old + sum >= 1);
//   end     done when no player bit is left or the counter reaches L; reward = sum over
//           fired rules of reward * popcount; done environments reload their initial rows.
// With rule application control (Sec. 2.1.1), the loaded rules of a batch only record their
// matches; group 0 (one lane per row) then filters them in index order — inhibition by the
// applied matches of earlier rules (rows OR-ed, then dilated over columns), a cap through a
// row-major prefix of per-row counts or, for the random index channel (Philox keys computed
// into LDS once per step), a radix select over a 256-bin LDS histogram — and the groups cast
// the filtered rules' votes and rewards before the write.
#include <algorithm>
#include <atomic>

#include "av_internal.h"
#include "philox.h"

namespace av {
namespace {

constexpr int kPad = 16;       // zero rows below the planes and above the match planes
constexpr int kMRows = kPad + 64;
constexpr int kBlock = 64;      // steps per block of actions, rewards and done flags

template <typename RowT>
__device__ inline RowT load_row(const void *base, size_t idx, int row_bytes) {
    if (row_bytes == 2) return static_cast<const uint16_t *>(base)[idx];
    if (row_bytes == 4) return static_cast<const uint32_t *>(base)[idx];
    return static_cast<RowT>(static_cast<const uint64_t *>(base)[idx]);
}

template <typename RowT>
__device__ inline void store_row(void *base, size_t idx, int row_bytes, RowT v) {
    if (row_bytes == 2) static_cast<uint16_t *>(base)[idx] = static_cast<uint16_t>(v);
    else if (row_bytes == 4) static_cast<uint32_t *>(base)[idx] = static_cast<uint32_t>(v);
    else static_cast<uint64_t *>(base)[idx] = static_cast<uint64_t>(v);
}

__device__ inline int popc(uint32_t v) { return __popc(v); }
__device__ inline int popc(uint64_t v) { return __popcll(v); }
__device__ inline int lowbit(uint32_t v) { return __ffs(v) - 1; }
__device__ inline int lowbit(uint64_t v) { return __ffsll(static_cast<unsigned long long>(v)) - 1; }
__device__ inline void lds_or(uint32_t *p, uint32_t v) { atomicOr(p, v); }
__device__ inline void lds_or(uint64_t *p, uint64_t v) {
    atomicOr(reinterpret_cast<unsigned long long *>(p), static_cast<unsigned long long>(v));
}
// value of lane `src` of this wave (byte address src * 4)
__device__ inline uint32_t from_lane(uint32_t v, int src) {
    return uint32_t(__builtin_amdgcn_ds_bpermute(src << 2, int(v)));
}
__device__ inline uint64_t from_lane(uint64_t v, int src) {
    return uint64_t(from_lane(uint32_t(v), src)) | (uint64_t(from_lane(uint32_t(v >> 32), src)) << 32);
}

template <typename RowT>
__device__ inline RowT low_mask(int bits) {
    return bits >= int(8 * sizeof(RowT)) ? ~RowT(0) : ((RowT(1) << bits) - 1);
}

// Does any lane of this thread's group (Hq consecutive lanes of the wave) hold a nonzero?
__device__ inline bool group_any(bool p, int Hq, int lane) {
    const unsigned long long bal = __builtin_amdgcn_ballot_w64(p);
    if (Hq >= 64) return bal != 0ull;
    const int base = lane & ~(Hq - 1);
    return ((bal >> base) & ((1ull << Hq) - 1ull)) != 0ull;
}

constexpr int kCountBits = 17;   // a cell-channel gets at most 256 rules x 16 x 16 votes

// Add the one-bit plane t to the bit-sliced counter cnt (bit k of every cell's count in
// cnt[k]); the carry ripples only as far as some lane of the group still carries.
template <typename RowT>
__device__ inline void count_add(RowT (&cnt)[kCountBits], RowT t, int Hq, int lane) {
#pragma unroll
    for (int k = 0; k < kCountBits; ++k) {
        if (!group_any(t != 0, Hq, lane)) break;
        const RowT carry = cnt[k] & t;
        cnt[k] ^= t;
        t = carry;
    }
}

// The exact write of channel c for this lane's row: counts every vote of every rule of the
// batch [rb, re) that fired (plus and minus separately, old value counted as a plus vote)
// and returns the cells where old + #plus > #minus, i.e. old + sum of votes >= 1.
template <typename RowT>
__device__ RowT exact_channel(int c, RowT old, int rb, int re, const int *fired,
                              const uint32_t *hdrw, const uint32_t *vent, const RowT *M, int y,
                              int Hq, int lane) {
    RowT pc[kCountBits], nc[kCountBits];
#pragma unroll
    for (int k = 0; k < kCountBits; ++k) pc[k] = nc[k] = 0;
    count_add<RowT>(pc, old, Hq, lane);
    constexpr int kHdrWords = sizeof(RuleHdr) / 4;
    for (int r = rb; r < re; ++r) {
        if (!fired[r]) continue;
        const uint32_t *hw = hdrw + r * kHdrWords;
        const RowT *Mr = M + size_t(r) * kMRows + kPad;
        const int voff = int(hw[5]), vcnt = int(hw[6]);
        for (int ev = 0; ev < vcnt; ++ev) {
            const uint32_t v = vent[voff + ev];
            if (int(v & 255) != c) continue;
            const int i = (v >> 8) & 255, j = (v >> 16) & 255;
            const RowT t = Mr[y - i] << j;
            if ((v >> 24) & 1) count_add<RowT>(pc, t, Hq, lane);
            else count_add<RowT>(nc, t, Hq, lane);
        }
    }
    RowT gt = 0, eq = ~RowT(0);
#pragma unroll
    for (int k = kCountBits - 1; k >= 0; --k) {
        gt |= eq & pc[k] & ~nc[k];
        eq &= ~(pc[k] ^ nc[k]);
    }
    return gt;
}

struct WaveLayout {
    int Hq;          // lanes per group (16, 32 or 64)
    int G;           // groups of Hq lanes
    int prog_lds;    // 1 if the rule program is copied into LDS
    int hdr_words, match_words, vote_words;
    int ctl_words;   // LDS words of the control scratch (0 without control)
};

// rowcnt [64], count [4], histogram [256], keys [H*W] (random order only)
int ctl_scratch_words(int H, int W, bool control, bool random) {
    return control ? 64 + 4 + 256 + (random ? H * W : 0) : 0;
}

// kMaxThreads: 1024 for 32-bit rows, 512 for 64-bit rows (their registers fit two waves per
// SIMD, not four)
template <typename RowT, int kMaxThreads>
__global__ void __launch_bounds__(kMaxThreads) wave_step(StepArgs a, WaveLayout L) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int H = a.H, W = a.W, C = a.C, C1 = C + 1, Hp = a.H + kPad, Hq = L.Hq, G = L.G;
    const int Rt = a.prog.rules_per_set;
    const int tid = threadIdx.x, nthreads = blockDim.x;
    const int g = tid / Hq, y = tid - g * Hq;
    const int lane = tid & 63;
    const int b = blockIdx.x;
    const int s = a.per_env ? b : 0;
    const bool row = y < H;
    const int ry = row ? y : H - 1;               // a safe row to read for idle lanes

    RowT *P = reinterpret_cast<RowT *>(lds);      // [C1][Hp]
    RowT *M = P + size_t(C1) * Hp;                // [Rt][kMRows]
    RowT *PL = M + size_t(Rt) * kMRows;           // [C1][64]
    RowT *MI = PL + size_t(C1) * 64;              // [C1][64]
    int *fired = reinterpret_cast<int *>(MI + size_t(C1) * 64);  // [Rt]
    int *red = fired + Rt;                        // [1] reward sum
    // Per block of 64 steps: the environment's actions, loaded at the block's first step,
    // and its rewards and done flags, stored after its last; a barrier waits for every
    // outstanding global access of the workgroup, so one load and one store per step would
    // each cost a memory latency per step.
    int *acts = red + 2;                          // [64]
    float *rblk = reinterpret_cast<float *>(acts + kBlock);    // [64]
    int *dblk = acts + 2 * kBlock;                // [64]
    int *rowcnt = acts + 3 * kBlock;              // control scratch (ctl_words words)
    int *ccnt = rowcnt + 64;
    int *hist = ccnt + 4;
    uint32_t *keys = reinterpret_cast<uint32_t *>(hist + 256);
    uint32_t *pcopy = reinterpret_cast<uint32_t *>(rowcnt + L.ctl_words);   // program copy

    const size_t words = size_t(C1) * Hp + size_t(Rt) * kMRows + size_t(2) * C1 * 64;
    for (size_t w = tid; w < words; w += nthreads) P[w] = 0;

    const uint32_t *ghdr = reinterpret_cast<const uint32_t *>(a.prog.hdr + size_t(s) * Rt);
    const uint32_t *gment = a.prog.match + size_t(s) * a.prog.match_stride;
    const uint32_t *gvent = a.prog.rvote + size_t(s) * a.prog.rvote_stride;
    const uint32_t *hdrw = ghdr, *ment = gment, *vent = gvent;
    if (L.prog_lds) {
        uint32_t *ph = pcopy, *pm = ph + L.hdr_words, *pv = pm + L.match_words;
        for (int w = tid; w < L.hdr_words; w += nthreads) ph[w] = ghdr[w];
        for (int w = tid; w < L.match_words; w += nthreads) pm[w] = gment[w];
        for (int w = tid; w < L.vote_words; w += nthreads) pv[w] = gvent[w];
        hdrw = ph;
        ment = pm;
        vent = pv;
    }
    __syncthreads();
    if (row)
        for (int c = g; c < C; c += G)
            P[c * Hp + y] = load_row<RowT>(a.state, (size_t(c) * a.B + b) * H + y, a.row_bytes);
    int t_env = a.t[b];
    // this workgroup's copy of the batch step number (read before the step loop's first
    // barrier; thread 0 stores it advanced by k after the last one)
    const uint64_t nbase = a.nctr[b];
    const RowT rowmask = low_mask<RowT>(W);
    constexpr int kHdrWords = sizeof(RuleHdr) / 4;

    // rewards and done flags of the block of 64 steps that ends before step k0
    auto flush = [&](int k0, int n) {
        if (tid < n) {
            a.rewards[size_t(k0 + tid) * a.B + b] = rblk[tid];
            a.done[size_t(k0 + tid) * a.B + b] = uint8_t(dblk[tid]);
        }
    };
    for (int k = 0; k < a.k; ++k) {
        for (int r = tid; r < Rt; r += nthreads) fired[r] = 0;
        if (tid == 0) *red = 0;
        const int kb = k & (kBlock - 1);
        if (kb == 0 && tid < kBlock && k + tid < a.k) acts[tid] = a.actions[size_t(k + tid) * a.B + b];
        __syncthreads();                          // previous step's rows are all written
        // the previous block's results (thread 0 wrote the last one after step k-1's final
        // barrier, so only after this one may other threads read it)
        if (kb == 0 && k > 0) flush(k - kBlock, kBlock);
        if (g == 0) {
            const int act = acts[kb];
            const RowT *Pp = P + kChPlayer * Hp;
            RowT f = 0;
            if (act == 1) f = Pp[ry + 1];         // row H is a zero pad row
            else if (act == 3) f = ry >= 1 ? Pp[ry - 1] : RowT(0);
            else if (act == 2) f = (Pp[ry] << 1) & rowmask;
            else if (act == 4) f = Pp[ry] >> 1;
            if (row) P[C * Hp + y] = f;
        }
        if (a.ctl.active && a.ctl.random) {
            // this step's random index channel, eight cells per Philox block
            const uint64_t n = nbase + uint64_t(k);
            for (int gi = tid; gi * 8 < H * W; gi += nthreads) {
                uint32_t u[8];
                philox_words(a.ctl.seed, n, uint64_t(b), 0, uint64_t(gi), u);
                for (int j = 0; j < 8 && gi * 8 + j < H * W; ++j)
                    keys[gi * 8 + j] = (u[j] & 0xFFFFF000u) | uint32_t(4095 - (gi * 8 + j));
            }
        }
        __syncthreads();

        // Rules in batches: all at once (parallel mode) or one at a time (sequential mode,
        // each rule matched on the map the previous ones left, force plane included).
        const int Cw = a.sequential ? C1 : C;     // planes the rules write
        int rsum = 0;
        for (int rb = 0, re = 0; rb < Rt; rb = re) {
            re = a.sequential ? rb + 1 : Rt;
            if (rb > 0) __syncthreads();          // the previous batch's rows are all written
            // group g takes rules rb+g, rb+g+G, ...; a rule that fired casts its votes at once
            for (int r = rb + g; r < re; r += G) {
                const uint32_t *hw = hdrw + r * kHdrWords;
                const int hn = int(hw[0]), hm = int(hw[1]), hreward = int(hw[2]);
                const int moff = int(hw[3]), mcnt = int(hw[4]), voff = int(hw[5]), vcnt = int(hw[6]);
                RowT acc = (row && y + hn <= H) ? low_mask<RowT>(W - hm + 1) : RowT(0);
                const uint32_t *en = ment + moff;
                int e = 0;
                for (; e + 4 <= mcnt && group_any(acc != 0, Hq, lane); e += 4) {
                    RowT v[4];
                    uint32_t q[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        q[u] = en[e + u];
                        v[u] = P[(q[u] & 255) * Hp + ry + ((q[u] >> 8) & 255)] >> ((q[u] >> 16) & 255);
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) acc &= ((q[u] >> 24) & 1) ? v[u] : RowT(~v[u]);
                }
                for (; e < mcnt && group_any(acc != 0, Hq, lane); ++e) {
                    const uint32_t q = en[e];
                    const RowT v = P[(q & 255) * Hp + ry + ((q >> 8) & 255)] >> ((q >> 16) & 255);
                    acc &= ((q >> 24) & 1) ? v : RowT(~v);
                }
                if (group_any(acc != 0, Hq, lane)) {
                    M[size_t(r) * kMRows + kPad + y] = acc;
                    if (y == 0) fired[r] = 1;
                    if (a.ctl.active && r >= kMoveRules) continue;   // filtered, then applied
                    rsum += hreward * popc(acc);
                    for (int ev = 0; ev < vcnt; ++ev) {
                        const uint32_t v = vent[voff + ev];
                        const int c = v & 255, i = (v >> 8) & 255, j = (v >> 16) & 255;
                        const RowT src = from_lane(acc, lane - (y >= i ? i : 0));
                        const RowT t = (y >= i) ? RowT(src << j) : RowT(0);
                        if (row && t) lds_or(((v >> 24) & 1 ? PL : MI) + c * 64 + y, t);
                    }
                }
            }
            __syncthreads();

            if (a.ctl.active) {
                // filter the batch's loaded rules in index order (group 0, lane = row)
                const int r0 = rb < kMoveRules ? kMoveRules : rb;
                for (int r = r0; r < re; ++r) {
                    if (!fired[r]) continue;                 // uniform: set before the last barrier
                    if (tid == 0) *ccnt = 0;
                    __syncthreads();
                    const size_t cr = size_t(s) * Rt + r;
                    const bool mine = g == 0 && row && fired[r];
                    RowT acc = mine ? M[size_t(r) * kMRows + kPad + y] : RowT(0);
                    if (mine && acc) {
                        const uint32_t *hw = hdrw + r * kHdrWords;
                        const int hn = int(hw[0]), hm = int(hw[1]);
                        const uint32_t *inh = a.ctl.inhibit + cr * a.ctl.words;
                        for (int w = 0; w < a.ctl.words; ++w) {
                            uint32_t bits = inh[w];
                            while (bits) {
                                const int q = w * 32 + __ffs(bits) - 1;
                                bits &= bits - 1;
                                if (!fired[q]) continue;
                                const uint32_t *qw = hdrw + q * kHdrWords;
                                const int nq = int(qw[0]), mq = int(qw[1]);
                                // anchors of q whose patch overlaps an hn x hm patch at row y
                                RowT o = 0;
                                const int ylo = y - nq + 1 < 0 ? 0 : y - nq + 1;
                                const int yhi = y + hn - 1 > H - 1 ? H - 1 : y + hn - 1;
                                for (int yy = ylo; yy <= yhi; ++yy) o |= M[size_t(q) * kMRows + kPad + yy];
                                RowT dil = o;
                                for (int d = 1; d < hm; ++d) dil |= o >> d;
                                for (int d = 1; d < mq; ++d) dil |= o << d;
                                acc &= ~dil;
                            }
                        }
                    }
                    if (g == 0) {
                        if (row && fired[r]) M[size_t(r) * kMRows + kPad + y] = acc;
                        if (y < 64) rowcnt[y] = row ? popc(acc) : 0;
                        if (acc) atomicAdd(ccnt, popc(acc));
                    }
                    __syncthreads();
                    const int lim = a.ctl.limit[cr];
                    if (lim > 0 && *ccnt > lim) {            // uniform: every thread reads ccnt
                        if (!a.ctl.random) {
                            if (mine) {
                                int before = 0;
                                for (int yy = 0; yy < y; ++yy) before += rowcnt[yy];
                                RowT keep = 0, rest = acc;
                                for (int kk = lim - before; kk > 0 && rest; --kk) {
                                    const RowT lb = rest & (~rest + 1);
                                    keep |= lb;
                                    rest ^= lb;
                                }
                                acc = keep;
                                M[size_t(r) * kMRows + kPad + y] = acc;
                            }
                        } else {
                            // radix select of the lim-th largest key among the matches
                            uint32_t prefix = 0, pmask = 0;
                            int need = lim;
                            for (int shift = 24; shift >= 0; shift -= 8) {
                                for (int i = tid; i < 256; i += nthreads) hist[i] = 0;
                                __syncthreads();
                                for (RowT rest = mine ? acc : RowT(0); rest; rest &= rest - 1) {
                                    const uint32_t key = keys[y * W + lowbit(rest)];
                                    if ((key & pmask) == prefix)
                                        atomicAdd(&hist[(key >> shift) & 255], 1);
                                }
                                __syncthreads();
                                int above = 0, d = 255;
                                for (; d > 0; --d) {
                                    const int cnt = hist[d];
                                    if (above + cnt >= need) break;
                                    above += cnt;
                                }
                                prefix |= uint32_t(d) << shift;
                                pmask |= 255u << shift;
                                need -= above;
                                __syncthreads();             // before the next pass clears hist
                            }
                            if (mine) {
                                RowT keep = 0;
                                for (RowT rest = acc; rest; rest &= rest - 1) {
                                    const int x = lowbit(rest);
                                    if (keys[y * W + x] >= prefix) keep |= RowT(1) << x;
                                }
                                acc = keep;
                                M[size_t(r) * kMRows + kPad + y] = acc;
                            }
                        }
                    }
                    __syncthreads();
                }
                // rewards and votes of the filtered loaded rules, group g taking rules g, g+G, ...
                for (int r = r0 + ((g - r0 % G + G) % G); r < re; r += G) {
                    if (!fired[r]) continue;
                    const uint32_t *hw = hdrw + r * kHdrWords;
                    const int hreward = int(hw[2]), voff = int(hw[5]), vcnt = int(hw[6]);
                    const RowT *Mr = M + size_t(r) * kMRows + kPad;
                    if (row) rsum += hreward * popc(Mr[y]);
                    for (int ev = 0; ev < vcnt; ++ev) {
                        const uint32_t v = vent[voff + ev];
                        const int c = v & 255, i = (v >> 8) & 255, j = (v >> 16) & 255;
                        const RowT t = RowT(Mr[y - i] << j);          // kPad zero rows above
                        if (row && t) lds_or(((v >> 24) & 1 ? PL : MI) + c * 64 + y, t);
                    }
                }
                __syncthreads();
            }

            // new rows: group g rewrites planes g, g+G, ... (each lane its own row)
            for (int c = g; c < Cw; c += G) {
                const RowT old = P[c * Hp + ry];
                const RowT pl = PL[c * 64 + y], mi = MI[c * 64 + y];
                RowT nw = (old | pl) & ~mi;
                const RowT mixed = pl & mi;
                if (group_any(mixed != 0, Hq, lane))
                    nw = exact_channel<RowT>(c, old, rb, re, fired, hdrw, vent, M, y, Hq, lane);
                if (row) P[c * Hp + y] = nw;
                PL[c * 64 + y] = 0;
                MI[c * 64 + y] = 0;
            }
        }
        if (rsum) atomicAdd(red, rsum);

        // episode end, reward, outputs, reset
        const bool anyp = __syncthreads_or(g == kChPlayer % G && row &&
                                           P[kChPlayer * Hp + y] != 0) != 0;
        t_env += 1;
        const bool d = !anyp || (a.L > 0 && t_env == a.L);
        if (d) t_env = 0;
        if (tid == 0) {
            rblk[kb] = float(*red);
            dblk[kb] = d ? 1 : 0;
        }
        if (d && row)
            for (int c = g; c < C; c += G)
                P[c * Hp + y] = load_row<RowT>(a.init, (size_t(c) * a.B + b) * H + y, a.row_bytes);
    }

    __syncthreads();
    if (a.k > 0) {
        const int n = ((a.k - 1) & (kBlock - 1)) + 1;
        flush(a.k - n, n);
    }
    if (row)
        for (int c = g; c < C; c += G)
            store_row<RowT>(a.state, (size_t(c) * a.B + b) * H + y, a.row_bytes, P[c * Hp + y]);
    if (tid == 0) {
        a.t[b] = t_env;
        a.nctr[b] = nbase + uint64_t(a.k);
    }
}

int rows_per_group(int H) { return H <= 16 ? 16 : (H <= 32 ? 32 : 64); }

// Groups per workgroup: the most for which the whole batch still fits the device's wave
// slots (8 waves per SIMD, 4 SIMDs per CU) at once, at most max_threads / Hq and at most the
// rule count rounded up to a power of two; else 4.  More groups match more of an
// environment's rules at once (c2, 1024 environments: 16 groups are 28-43 % faster than 4),
// but past the wave slots they only add rounds of workgroups (c4 on this engine, 16384
// environments: 36 against 18 us per step; c3, 4096: 8 groups 10 % slower than 4).
int wave_groups(int B, int Hq, int rules, int max_threads) {
    const long long slots = device_wave_slots();
    if (slots <= 0) return 4;
    int cap = 4;
    while (cap < rules) cap *= 2;
    for (int G = std::min(max_threads / Hq, cap); G > 4; G /= 2)
        if (static_cast<long long>(B) * (G * Hq / 64) <= slots) return G;
    return 4;
}

size_t wave_base_bytes(int H, int W, int C, int rules_per_set) {
    const size_t rowb = W <= 32 ? 4 : 8;
    return (size_t(C + 1) * (H + kPad) + size_t(rules_per_set) * kMRows + size_t(2) * (C + 1) * 64) *
               rowb +
           sizeof(int) * (size_t(rules_per_set) + 2 + 3 * kBlock);
}

}  // namespace

long long device_wave_slots() {
    static std::atomic<int> cus[64];                 // per device, 0 until first asked
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int n = cus[dev].load(std::memory_order_relaxed);
    if (!n) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            return 0;
        cus[dev].store(n, std::memory_order_relaxed);
    }
    return 32LL * n;
}

size_t wave_lds_bytes(int H, int W, int C, int rules_per_set, bool control, bool random) {
    return wave_base_bytes(H, W, C, rules_per_set) +
           sizeof(int) * size_t(ctl_scratch_words(H, W, control, random));
}

hipError_t launch_wave_step(const StepArgs &a, hipStream_t s) {
    WaveLayout L;
    L.Hq = rows_per_group(a.H);
    const int max_threads = a.W <= 32 ? 1024 : 512;
    L.G = wave_groups(a.B, L.Hq, a.prog.rules_per_set, max_threads);
    L.hdr_words = int(a.prog.rules_per_set * (sizeof(RuleHdr) / 4));
    L.match_words = a.prog.match_stride;
    L.vote_words = a.prog.rvote_stride;
    L.ctl_words = ctl_scratch_words(a.H, a.W, a.ctl.active != 0, a.ctl.random != 0);
    const size_t base = wave_lds_bytes(a.H, a.W, a.C, a.prog.rules_per_set, a.ctl.active != 0,
                                       a.ctl.random != 0);
    const size_t prog = size_t(L.hdr_words + L.match_words + L.vote_words) * 4;
    // the copy pays for itself over a launch of many steps, not over one
    L.prog_lds = a.k >= 16 && base + prog <= size_t(kLdsBudget) ? 1 : 0;
    const size_t lds = base + (L.prog_lds ? prog : 0);
    const int threads = L.G * L.Hq;
    if (a.W <= 32)
        hipLaunchKernelGGL((wave_step<uint32_t, 1024>), dim3(a.B), dim3(threads), lds, s, a, L);
    else
        hipLaunchKernelGGL((wave_step<uint64_t, 512>), dim3(a.B), dim3(threads), lds, s, a, L);
    return hipGetLastError();
}

}  // namespace av
