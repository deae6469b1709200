// Generic step kernel and the pack / unpack kernels.
//
// Generic step: a workgroup holds G environments; thread (g, y) owns row y of environment
// g in every plane.  The C + 1 planes (stored channels plus the force plane) and one match
// plane per rule live in LDS for all k steps of the launch; rows are 32-bit words for
// W <= 32 and 64-bit words for W <= 64, one bit per cell, bit x = column x.
//
// Per step (paper Sec. 2.1, Sec. 2.1.1, Sec. 2.2.1):
//   force     F[y] = the player row shifted one cell toward the action's direction;
//   match     M_r[y] = AND over the rule's specified input entries of the plane row
//             y + i shifted right by j (bit x then holds cell x + j), complemented for
//             must-be-0 entries, masked to anchors where the pattern lies on the map;
//   control   (optional, Sec. 2.1.1) per loaded rule in index order: drop matches whose
//             patch overlaps an applied match of an inhibiting earlier rule, then keep the
//             `limit` matches with the largest index-channel value (radix select over the
//             32-bit keys, 8 bits per pass, through an LDS histogram per environment);
//   reward    sum over rules of reward_r * popcount(M_r), reduced per environment;
//   (order)   all rules match the same map (parallel mode), or in sequential mode each rule
//             is matched, and its votes applied, before the next one;
//   write     per channel, the OR of +1 votes and of -1 votes (match planes shifted back
//             by (i, j)); cells that got votes of one sign take that sign's value, cells
//             with both signs count the votes exactly: new = (old + sum >= 1);
//   end       done when no player bit is left or the counter reaches L; done
//             environments reload their initial rows.
#include <algorithm>

#include "av_internal.h"
#include "philox.h"

namespace av {
namespace {

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

template <typename RowT>
__device__ inline RowT low_mask(int bits) {
    return bits >= int(8 * sizeof(RowT)) ? ~RowT(0) : ((RowT(1) << bits) - 1);
}

// Index-channel value of cell pos: row-major rank 4095 - pos, or, for the random channel,
// the high 20 bits of the cell's Philox word above that rank (keys never tie).
__device__ inline uint32_t rank_key(int pos) { return uint32_t(4095 - pos); }

template <typename RowT>
__global__ void __launch_bounds__(256) generic_step(StepArgs a, int G) {
    extern __shared__ __align__(16) unsigned char lds[];
    const int H = a.H, W = a.W, C = a.C, C1 = C + 1;
    const int Rt = a.prog.rules_per_set;
    const int tid = threadIdx.x;
    const int g = tid / H, y = tid - (tid / H) * H;
    const int b = blockIdx.x * G + g;
    const bool live = g < G && b < a.B;
    const int s = a.per_env ? b : 0;

    RowT *planes = reinterpret_cast<RowT *>(lds);        // [G][C1][H]
    RowT *M = planes + size_t(G) * C1 * H;               // [G][Rt][H]
    int *red = reinterpret_cast<int *>(M + size_t(G) * Rt * H);  // [G] reward sums
    int *anyp = red + G;                                  // [G] player bits left
    int *dflag = anyp + G;                                // [G] done this step
    int *cnt = dflag + G;                                 // [G] matches of one rule
    int *hist = cnt + G;                                  // [G][256] radix histogram
    uint32_t *keys = reinterpret_cast<uint32_t *>(hist + (a.ctl.active ? G * 256 : 0));
    const int HW = H * W;                                 // keys: [G][H*W] random channel

    const RowT rowmask = low_mask<RowT>(W);
    RowT *my = planes + size_t(g) * C1 * H;               // this env's planes
    RowT *myM = M + size_t(g) * Rt * H;

    if (live)
        for (int c = 0; c < C; ++c)
            my[c * H + y] = load_row<RowT>(a.state, (size_t(c) * a.B + b) * H + y, a.row_bytes);
    int t_env = (live && y == 0) ? a.t[b] : 0;
    // this workgroup's copy of the batch step number (read here, before the first barrier;
    // thread 0 stores it advanced by k after the last one)
    const uint64_t nbase = a.nctr[blockIdx.x];

    const RuleHdr *hdr = a.prog.hdr + size_t(s) * Rt;
    const uint32_t *ment = a.prog.match + size_t(s) * a.prog.match_stride;
    const VoteList *vl = a.prog.votes + size_t(s) * C1;
    const uint32_t *vent = a.prog.vote + size_t(s) * a.prog.vote_stride;

    for (int k = 0; k < a.k; ++k) {
        if (tid < G) { red[tid] = 0; anyp[tid] = 0; }
        __syncthreads();

        // force plane from the player plane and the action
        if (live) {
            const int act = a.actions[size_t(k) * a.B + b];
            const RowT *P = my + kChPlayer * H;
            RowT f = 0;
            if (act == 1) f = (y + 1 < H) ? P[y + 1] : RowT(0);
            else if (act == 3) f = (y >= 1) ? P[y - 1] : RowT(0);
            else if (act == 2) f = (P[y] << 1) & rowmask;
            else if (act == 4) f = P[y] >> 1;
            my[C * H + y] = f;
        }
        if (a.ctl.active && a.ctl.random && live) {
            // this step's random index channel, eight cells per Philox block
            const uint64_t n = nbase + uint64_t(k);
            for (int gi = y; gi * 8 < HW; gi += H) {
                uint32_t u[8];
                philox_words(a.ctl.seed, n, uint64_t(b), 0, uint64_t(gi), u);
                for (int j = 0; j < 8 && gi * 8 + j < HW; ++j) {
                    const int pos = gi * 8 + j;
                    keys[size_t(g) * HW + pos] = (u[j] & 0xFFFFF000u) | rank_key(pos);
                }
            }
        }
        __syncthreads();

        // Rules in batches: all of them at once (parallel mode) or one at a time
        // (sequential mode, each rule matched on the map the previous ones left).
        int rsum = 0;
        for (int r0 = 0, r1 = 0; r0 < Rt; r0 = r1) {
            r1 = a.sequential ? r0 + 1 : Rt;
            if (r0 > 0) __syncthreads();      // the previous batch's rows are all written
            if (live) {
                for (int r = r0; r < r1; ++r) {
                    const RuleHdr h = hdr[r];
                    RowT acc = (y + h.n <= H) ? low_mask<RowT>(W - h.m + 1) : RowT(0);
                    for (int e = 0; e < h.match_cnt && acc; ++e) {
                        const uint32_t en = ment[h.match_off + e];
                        const int c = en & 255, i = (en >> 8) & 255, j = (en >> 16) & 255;
                        const RowT v = my[c * H + y + i] >> j;
                        acc &= ((en >> 24) & 1) ? v : RowT(~v);
                    }
                    myM[r * H + y] = acc;
                    if (!a.ctl.active) rsum += h.reward * popc(acc);
                }
            }
            __syncthreads();

            if (a.ctl.active) {
                // loaded rules of the batch in index order: inhibition, then the limit
                for (int r = r0 < kMoveRules ? kMoveRules : r0; r < r1; ++r) {
                    if (tid < G) cnt[tid] = 0;
                    const size_t cr = size_t(s) * Rt + r;
                    RowT acc = live ? myM[r * H + y] : RowT(0);
                    if (live && acc) {
                        const RuleHdr h = hdr[r];
                        const uint32_t *inh = a.ctl.inhibit + cr * a.ctl.words;
                        for (int w = 0; w < a.ctl.words; ++w) {
                            uint32_t bits = inh[w];
                            while (bits) {
                                const int q = w * 32 + __ffs(bits) - 1;
                                bits &= bits - 1;
                                const int nq = hdr[q].n, mq = hdr[q].m;
                                // anchors of q whose patch overlaps an n x m patch at row y:
                                // rows y - nq + 1 .. y + n - 1, columns x - mq + 1 .. x + m - 1
                                RowT o = 0;
                                const int ylo = y - nq + 1 < 0 ? 0 : y - nq + 1;
                                const int yhi = y + h.n - 1 > H - 1 ? H - 1 : y + h.n - 1;
                                for (int yy = ylo; yy <= yhi; ++yy) o |= myM[q * H + yy];
                                RowT dil = o;
                                for (int d = 1; d < h.m; ++d) dil |= o >> d;
                                for (int d = 1; d < mq; ++d) dil |= o << d;
                                acc &= ~dil;
                            }
                        }
                    }
                    __syncthreads();                 // cnt cleared; rows q < r all read
                    if (live) {
                        myM[r * H + y] = acc;
                        atomicAdd(&cnt[g], popc(acc));
                    }
                    __syncthreads();
                    const int lim = live ? a.ctl.limit[cr] : 0;
                    const bool sel = live && lim > 0 && cnt[g] > lim;
                    if (__syncthreads_or(sel)) {
                        // radix select of the lim-th largest key among the matches
                        uint32_t prefix = 0, pmask = 0;
                        int need = lim;
                        for (int shift = 24; shift >= 0; shift -= 8) {
                            for (int i = tid; i < G * 256; i += blockDim.x) hist[i] = 0;
                            __syncthreads();
                            if (sel) {
                                RowT rest = acc;
                                while (rest) {
                                    const int x = lowbit(rest);
                                    rest &= rest - 1;
                                    const int pos = y * W + x;
                                    const uint32_t key = a.ctl.random ? keys[size_t(g) * HW + pos]
                                                                      : rank_key(pos);
                                    if ((key & pmask) == prefix)
                                        atomicAdd(&hist[g * 256 + ((key >> shift) & 255)], 1);
                                }
                            }
                            __syncthreads();
                            if (sel) {
                                int above = 0, d = 255;
                                for (; d > 0; --d) {
                                    const int c = hist[g * 256 + d];
                                    if (above + c >= need) break;
                                    above += c;
                                }
                                prefix |= uint32_t(d) << shift;
                                pmask |= 255u << shift;
                                need -= above;
                            }
                            __syncthreads();         // before the next pass clears hist
                        }
                        if (sel) {
                            RowT rest = acc, keep = 0;
                            while (rest) {
                                const int x = lowbit(rest);
                                rest &= rest - 1;
                                const int pos = y * W + x;
                                const uint32_t key = a.ctl.random ? keys[size_t(g) * HW + pos]
                                                                  : rank_key(pos);
                                if (key >= prefix) keep |= RowT(1) << x;
                            }
                            myM[r * H + y] = keep;
                        }
                    }
                }
                if (live)
                    for (int r = r0; r < r1; ++r) rsum += hdr[r].reward * popc(myM[r * H + y]);
                __syncthreads();
            }

            // votes of this batch and clamp, one channel at a time; each thread rewrites
            // only its own row
            if (live) {
                for (int c = 0; c < C1; ++c) {
                    const VoteList L = vl[c];
                    RowT plus = 0, minus = 0;
                    for (int e = 0; e < L.cnt; ++e) {
                        const uint32_t v = vent[L.off + e];
                        const int r = v & 255, i = (v >> 8) & 255, j = (v >> 16) & 255;
                        if (r < r0 || r >= r1 || y < i) continue;
                        const RowT mv = myM[r * H + y - i] << j;
                        if ((v >> 24) & 1) plus |= mv; else minus |= mv;
                    }
                    const RowT old = my[c * H + y];
                    RowT nw = (old | plus) & ~minus;
                    RowT mixed = plus & minus;
                    while (mixed) {       // cells with votes of both signs: count exactly
                        const int x = lowbit(mixed);
                        mixed &= mixed - 1;
                        int sum = int((old >> x) & 1);
                        for (int e = 0; e < L.cnt; ++e) {
                            const uint32_t v = vent[L.off + e];
                            const int r = v & 255, i = (v >> 8) & 255, j = (v >> 16) & 255;
                            if (r < r0 || r >= r1 || y < i || x < j) continue;
                            if ((myM[r * H + y - i] >> (x - j)) & 1) sum += ((v >> 24) & 1) ? 1 : -1;
                        }
                        nw = (nw & ~(RowT(1) << x)) | (RowT(sum >= 1 ? 1 : 0) << x);
                    }
                    my[c * H + y] = nw;
                }
            }
        }
        if (live) {
            if (my[kChPlayer * H + y]) atomicOr(&anyp[g], 1);
            atomicAdd(&red[g], rsum);
        }
        __syncthreads();

        if (live && y == 0) {
            t_env += 1;
            const int d = (anyp[g] == 0) || (a.L > 0 && t_env == a.L);
            if (d) t_env = 0;
            a.rewards[size_t(k) * a.B + b] = float(red[g]);
            a.done[size_t(k) * a.B + b] = uint8_t(d);
            dflag[g] = d;
        }
        __syncthreads();
        if (live && dflag[g])
            for (int c = 0; c < C; ++c)
                my[c * H + y] = load_row<RowT>(a.init, (size_t(c) * a.B + b) * H + y, a.row_bytes);
    }

    if (live) {
        for (int c = 0; c < C; ++c)
            store_row<RowT>(a.state, (size_t(c) * a.B + b) * H + y, a.row_bytes, my[c * H + y]);
        if (y == 0) a.t[b] = t_env;
    }
    if (tid == 0) a.nctr[blockIdx.x] = nbase + uint64_t(a.k);
}

// uint8 [B][C][H][W] -> packed rows [C][B][H]; one thread per row.
__global__ void pack_rows(const uint8_t *src, void *dst, void *dst2, int B, int C, int H, int W,
                          int row_bytes) {
    const size_t row = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const size_t rows = size_t(B) * C * H;
    if (row >= rows) return;
    const int y = int(row % H);
    const size_t cb = row / H;
    const int b = int(cb % B), c = int(cb / B);
    const uint8_t *p = src + ((size_t(b) * C + c) * H + y) * W;
    uint64_t v = 0;
    for (int x = 0; x < W; ++x) v |= uint64_t(p[x] != 0) << x;
    store_row<uint64_t>(dst, row, row_bytes, v);
    if (dst2) store_row<uint64_t>(dst2, row, row_bytes, v);
}

// t[0..B) = 0 (when t is given) and nctr[0..n) = value, or nctr[0] when broadcasting
// (thread 0 then leaves nctr[0] alone, so every thread reads the same value).
__global__ void fill_counters(int32_t *t, int B, uint64_t *nctr, int n, int broadcast,
                              uint64_t value) {
    const int i = int(blockIdx.x * blockDim.x + threadIdx.x);
    if (t && i < B) t[i] = 0;
    if (i < n) {
        if (!broadcast) nctr[i] = value;
        else if (i > 0) nctr[i] = nctr[0];
    }
}

// packed rows [C][B][H] -> uint8 [B][C][H][W]; one thread per row.
__global__ void unpack_rows(const void *src, uint8_t *dst, int B, int C, int H, int W,
                            int row_bytes) {
    const size_t row = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const size_t rows = size_t(B) * C * H;
    if (row >= rows) return;
    const int y = int(row % H);
    const size_t cb = row / H;
    const int b = int(cb % B), c = int(cb / B);
    const uint64_t v = load_row<uint64_t>(src, row, row_bytes);
    uint8_t *p = dst + ((size_t(b) * C + c) * H + y) * W;
    for (int x = 0; x < W; ++x) p[x] = uint8_t((v >> x) & 1);
}

}  // namespace

size_t generic_env_lds_bytes(int H, int W, int C, int rules_per_set, bool control,
                             bool random) {
    const size_t rowb = W <= 32 ? 4 : 8;
    size_t bytes = size_t(C + 1 + rules_per_set) * H * rowb + 4 * sizeof(int);
    if (control) bytes += 256 * sizeof(int) + (random ? size_t(H) * W * sizeof(uint32_t) : 0);
    return bytes;
}

hipError_t launch_generic_step(const StepArgs &a, int G, hipStream_t s) {
    const int threads = G * a.H;
    const int blocks = (a.B + G - 1) / G;
    const size_t lds = size_t(G) * generic_env_lds_bytes(a.H, a.W, a.C, a.prog.rules_per_set,
                                                         a.ctl.active, a.ctl.random);
    if (a.W <= 32)
        hipLaunchKernelGGL(generic_step<uint32_t>, dim3(blocks), dim3(threads), lds, s, a, G);
    else
        hipLaunchKernelGGL(generic_step<uint64_t>, dim3(blocks), dim3(threads), lds, s, a, G);
    return hipGetLastError();
}

hipError_t launch_pack(const uint8_t *src, void *dst, void *dst2, int B, int C, int H, int W,
                       int row_bytes, hipStream_t s) {
    const size_t rows = size_t(B) * C * H;
    const int threads = 256;
    const unsigned blocks = unsigned((rows + threads - 1) / threads);
    hipLaunchKernelGGL(pack_rows, dim3(blocks), dim3(threads), 0, s, src, dst, dst2, B, C, H, W,
                       row_bytes);
    return hipGetLastError();
}

hipError_t launch_fill_counters(int32_t *t, int B, uint64_t *nctr, int n, int broadcast,
                                uint64_t value, hipStream_t s) {
    const int m = std::max(t ? B : 0, n);
    if (m <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_counters, dim3(unsigned((m + 255) / 256)), dim3(256), 0, s, t, B, nctr,
                       n, broadcast, value);
    return hipGetLastError();
}

hipError_t launch_unpack(const void *src, uint8_t *dst, int B, int C, int H, int W,
                         int row_bytes, hipStream_t s) {
    const size_t rows = size_t(B) * C * H;
    const int threads = 256;
    const unsigned blocks = unsigned((rows + threads - 1) / threads);
    hipLaunchKernelGGL(unpack_rows, dim3(blocks), dim3(threads), 0, s, src, dst, B, C, H, W,
                       row_bytes);
    return hipGetLastError();
}

}  // namespace av
