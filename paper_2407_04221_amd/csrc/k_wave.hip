// wave engine: one environment per 64-lane workgroup; lane y owns map row y (H <= 64).
//
// With one environment per wave, the environment's rule program is wave-uniform even
// when every environment has its own rules: rule headers and entries come in through
// scalar loads, and a rule that matches nowhere in the map costs one ballot.
//
// LDS (one environment):
//   planes  [C+1][H+16] rows: the map and the force plane; 16 zero rows below the map let
//           a lane read row y+i of any pattern without a bounds test
//   match   [R+4][16+64] rows: match planes of the rules that fired, 16 zero rows on top
//           so that row y-i of a vote is always a valid read
//   plus, minus [C][64] rows: per channel, OR of the +1 and of the -1 votes
//   fired   [R+4] indices of the rules that fired this step
// Rows are 32-bit words for W <= 32, 64-bit for W <= 64; bit x = column x.
//
// Per step (paper Sec. 2.1, Sec. 2.1.1, Sec. 2.2.1):
//   force   F[y] = the player row moved one cell toward the action;
//   match   for every rule, AND over its specified entries (rarest first) of plane row
//           y+i shifted right by j (complemented for must-be-0), within the valid-anchor
//           mask; the wave leaves the rule as soon as no anchor survives;
//   votes   for the rules that fired, each nonzero K_O = O - I entry ORs the match plane
//           moved by (i, j) into the plus or minus accumulator of its channel (LDS atomic OR);
//   write   new = (old | plus) & ~minus where no cell got both signs; a row with mixed
//           cells counts their votes exactly: new = (old + sum >= 1);
//   end     done when no player bit is left or the counter reaches L; reward = sum over
//           fired rules of reward * popcount; done environments reload their initial rows.
#include "av_internal.h"

namespace av {
namespace {

constexpr int kPad = 16;       // zero rows below the planes and above the match planes
constexpr int kMRows = kPad + 64;

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

template <typename RowT>
__device__ inline RowT low_mask(int bits) {
    return bits >= int(8 * sizeof(RowT)) ? ~RowT(0) : ((RowT(1) << bits) - 1);
}

__device__ inline bool wave_any(bool p) { return __builtin_amdgcn_ballot_w64(p) != 0ull; }

__device__ inline int wave_sum(int v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

template <typename RowT>
__global__ void __launch_bounds__(64) wave_step(StepArgs a) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int H = a.H, W = a.W, C = a.C, C1 = C + 1, Hp = a.H + kPad;
    const int Rt = a.prog.rules_per_set;
    const int y = threadIdx.x;
    const int b = blockIdx.x;
    const int s = a.per_env ? b : 0;
    const bool row = y < H;
    const int ry = row ? y : H - 1;               // a safe row to read for idle lanes

    RowT *P = reinterpret_cast<RowT *>(lds);      // [C1][Hp]
    RowT *M = P + size_t(C1) * Hp;                // [Rt][kMRows]
    RowT *PL = M + size_t(Rt) * kMRows;           // [C][64]
    RowT *MI = PL + size_t(C) * 64;               // [C][64]
    int *fired = reinterpret_cast<int *>(MI + size_t(C) * 64);

    const size_t words = size_t(C1) * Hp + size_t(Rt) * kMRows + size_t(2) * C * 64;
    for (size_t w = y; w < words; w += 64) P[w] = 0;
    __syncthreads();
    if (row)
        for (int c = 0; c < C; ++c)
            P[c * Hp + y] = load_row<RowT>(a.state, (size_t(c) * a.B + b) * H + y, a.row_bytes);
    int t_env = a.t[b];

    const RuleHdr *hdr = a.prog.hdr + size_t(s) * Rt;
    const uint32_t *ment = a.prog.match + size_t(s) * a.prog.match_stride;
    const uint32_t *vent = a.prog.rvote + size_t(s) * a.prog.rvote_stride;
    const RowT rowmask = low_mask<RowT>(W);

    for (int k = 0; k < a.k; ++k) {
        __syncthreads();                          // previous step's rows are all written
        const int act = a.actions[size_t(k) * a.B + b];
        {
            const RowT *Pp = P + kChPlayer * Hp;
            RowT f = 0;
            if (act == 1) f = Pp[ry + 1];         // row H is a zero pad row
            else if (act == 3) f = ry >= 1 ? Pp[ry - 1] : RowT(0);
            else if (act == 2) f = (Pp[ry] << 1) & rowmask;
            else if (act == 4) f = Pp[ry] >> 1;
            if (row) P[C * Hp + y] = f;
        }
        __syncthreads();

        // match every rule on the same map; remember the ones that fired
        int rsum = 0, nf = 0;
        for (int r = 0; r < Rt; ++r) {
            const RuleHdr h = hdr[r];
            RowT acc = (row && y + h.n <= H) ? low_mask<RowT>(W - h.m + 1) : RowT(0);
            const uint32_t *en = ment + h.match_off;
            int e = 0;
            for (; e + 4 <= h.match_cnt && wave_any(acc != 0); e += 4) {
                RowT v[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const uint32_t q = en[e + u];
                    v[u] = P[(q & 255) * Hp + ry + ((q >> 8) & 255)] >> ((q >> 16) & 255);
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) acc &= ((en[e + u] >> 24) & 1) ? v[u] : RowT(~v[u]);
            }
            for (; e < h.match_cnt && wave_any(acc != 0); ++e) {
                const uint32_t q = en[e];
                const RowT v = P[(q & 255) * Hp + ry + ((q >> 8) & 255)] >> ((q >> 16) & 255);
                acc &= ((q >> 24) & 1) ? v : RowT(~v);
            }
            if (wave_any(acc != 0)) {
                M[size_t(r) * kMRows + kPad + y] = acc;
                if (y == 0) fired[nf] = r;
                ++nf;
                rsum += h.reward * popc(acc);
            }
        }
        __syncthreads();

        // votes of the rules that fired
        for (int q = 0; q < nf; ++q) {
            const int r = __builtin_amdgcn_readfirstlane(fired[q]);
            const RuleHdr h = hdr[r];
            const RowT *Mr = M + size_t(r) * kMRows + kPad;
            for (int e = 0; e < h.vote_cnt; ++e) {
                const uint32_t v = vent[h.vote_off + e];
                const int c = v & 255, i = (v >> 8) & 255, j = (v >> 16) & 255;
                const RowT t = Mr[y - i] << j;
                if (row && t) lds_or(((v >> 24) & 1 ? PL : MI) + c * 64 + y, t);
            }
        }
        __syncthreads();

        // new rows, one channel at a time (each lane rewrites only its own row)
        for (int c = 0; c < C; ++c) {
            const RowT old = P[c * Hp + ry];
            const RowT pl = PL[c * 64 + y], mi = MI[c * 64 + y];
            RowT nw = (old | pl) & ~mi;
            RowT mixed = pl & mi;
            if (wave_any(mixed != 0)) {
                while (mixed) {              // cells with votes of both signs: count exactly
                    const int x = lowbit(mixed);
                    mixed &= mixed - 1;
                    int sum = int((old >> x) & 1);
                    for (int q = 0; q < nf; ++q) {
                        const int r = fired[q];
                        const RuleHdr h = hdr[r];
                        const RowT *Mr = M + size_t(r) * kMRows + kPad;
                        for (int e = 0; e < h.vote_cnt; ++e) {
                            const uint32_t v = vent[h.vote_off + e];
                            const int i = (v >> 8) & 255, j = (v >> 16) & 255;
                            if (int(v & 255) != c || x < j) continue;
                            if ((Mr[y - i] >> (x - j)) & 1) sum += ((v >> 24) & 1) ? 1 : -1;
                        }
                    }
                    nw = (nw & ~(RowT(1) << x)) | (RowT(sum >= 1 ? 1 : 0) << x);
                }
            }
            if (row) P[c * Hp + y] = nw;
            PL[c * 64 + y] = 0;
            MI[c * 64 + y] = 0;
        }

        // episode end, reward, outputs, reset
        const bool anyp = wave_any(row && P[kChPlayer * Hp + y] != 0);
        t_env += 1;
        const bool d = !anyp || (a.L > 0 && t_env == a.L);
        if (d) t_env = 0;
        int reward = 0;
        if (a.prog.any_reward && nf > 0) reward = wave_sum(rsum);
        if (y == 0) {
            a.rewards[size_t(k) * a.B + b] = float(reward);
            a.done[size_t(k) * a.B + b] = uint8_t(d);
        }
        if (d && row)
            for (int c = 0; c < C; ++c)
                P[c * Hp + y] = load_row<RowT>(a.init, (size_t(c) * a.B + b) * H + y, a.row_bytes);
    }

    if (row)
        for (int c = 0; c < C; ++c)
            store_row<RowT>(a.state, (size_t(c) * a.B + b) * H + y, a.row_bytes, P[c * Hp + y]);
    if (y == 0) a.t[b] = t_env;
}

}  // namespace

size_t wave_lds_bytes(int H, int W, int C, int rules_per_set) {
    const size_t rowb = W <= 32 ? 4 : 8;
    return (size_t(C + 1) * (H + kPad) + size_t(rules_per_set) * kMRows + size_t(2) * C * 64) * rowb +
           sizeof(int) * size_t(rules_per_set);
}

hipError_t launch_wave_step(const StepArgs &a, hipStream_t s) {
    const size_t lds = wave_lds_bytes(a.H, a.W, a.C, a.prog.rules_per_set);
    if (a.W <= 32)
        hipLaunchKernelGGL(wave_step<uint32_t>, dim3(a.B), dim3(64), lds, s, a);
    else
        hipLaunchKernelGGL(wave_step<uint64_t>, dim3(a.B), dim3(64), lds, s, a);
    return hipGetLastError();
}

}  // namespace av
