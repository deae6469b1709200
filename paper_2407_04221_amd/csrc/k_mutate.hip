// Batched mutation operators (paper Sec. 2.2.1 and the Fig. 2b caption): environments are
// mutated by flipping bits of their initial multi-hot maps, by changing entries of their
// rules' input and output patterns, and by redrawing rule rewards.  Every individual of a
// population is mutated independently; each thread owns one Philox block (eight 32-bit
// words) and the elements those words decide, so the kernels are embarrassingly parallel,
// read and write each element once, and may run in place.
//
//   maps     element e = (c * H + y) * W + x of individual k: one word (stream 1, word e);
//            flip iff channel c is allowed and the word is below the flip threshold;
//   entries  element e = (((r * 2 + io) * (C+1) + c) * mh + i) * mw + j of set s: two words
//            (stream 2, words 2e and 2e + 1); inside the rule's n x m and on an allowed
//            channel, change iff word 2e is below the entry threshold, to the lower (word
//            2e + 1 even) or higher (odd) of the two other values of {-1, 0, 1};
//   rewards  rule r of set s: stream 3, words 2r (redraw iff below the reward threshold)
//            and 2r + 1 (new reward lo + word mod (hi - lo + 1)).
#include <algorithm>

#include "av_internal.h"
#include "philox.h"

namespace av {
namespace {

// Thread t of a launch covers Philox block t % blocks_per of individual k0 + t / blocks_per
// (32-bit index arithmetic: the launcher splits populations into chunks that fit).
__global__ void __launch_bounds__(256) mutate_maps_kernel(const uint8_t *src, uint8_t *dst,
                                                          int k0, int nk, int per, int plane,
                                                          int blocks_per, MutateArgs m) {
    const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= uint32_t(nk) * uint32_t(blocks_per)) return;
    const int kk = int(t / uint32_t(blocks_per));
    const int blk = int(t - uint32_t(kk) * uint32_t(blocks_per));
    const int k = k0 + kk;
    uint32_t w[8];
    philox_words(m.seed, m.generation, uint64_t(k), 1, uint64_t(blk), w);
    const int e0 = blk * 8;
    int c = e0 / plane, next = (c + 1) * plane;       // channel of element e, and its end
    const uint8_t *s = src + size_t(k) * per + e0;
    uint8_t *d = dst + size_t(k) * per + e0;
    uint32_t flips = 0;                               // bit j: element e0 + j flips
    for (int j = 0; j < 8; ++j) {
        while (e0 + j >= next) { ++c; next += plane; }
        flips |= uint32_t(((m.map_channels >> c) & 1u) && w[j] < m.map_flip_p32) << j;
    }
    if (e0 + 8 <= per && ((reinterpret_cast<uintptr_t>(s) | reinterpret_cast<uintptr_t>(d)) & 7) == 0) {
        // eight whole bytes, aligned: one 64-bit load and store
        const uint64_t v = *reinterpret_cast<const uint64_t *>(s);
        uint64_t out = 0;
        for (int j = 0; j < 8; ++j)
            out |= uint64_t((((v >> (8 * j)) & 0xFF) != 0) ^ ((flips >> j) & 1u)) << (8 * j);
        *reinterpret_cast<uint64_t *>(d) = out;
    } else {
        for (int j = 0; j < 8 && e0 + j < per; ++j)
            d[j] = uint8_t(s[j] != 0) ^ uint8_t((flips >> j) & 1u);
    }
}

__device__ inline int8_t other_value(int8_t old, bool higher) {
    const int v = (old == -1 || old == 0) ? old : 1;
    return int8_t(higher ? (v == 1 ? 0 : 1) : (v == -1 ? 0 : -1));
}

__global__ void __launch_bounds__(256) mutate_entries_kernel(
    const int32_t *shape, const int8_t *in_src, const int8_t *out_src, int8_t *in_dst,
    int8_t *out_dst, int s0, int ns, int R, int C1, int mh, int mw, int blocks_per,
    MutateArgs m) {
    const uint32_t t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= uint32_t(ns) * uint32_t(blocks_per)) return;
    const int ss = int(t / uint32_t(blocks_per));
    const int blk = int(t - uint32_t(ss) * uint32_t(blocks_per));
    const int s = s0 + ss;
    const int per = R * 2 * C1 * mh * mw;
    const int pat = C1 * mh * mw;
    uint32_t w[8];
    philox_words(m.seed, m.generation, uint64_t(s), 2, uint64_t(blk), w);
    for (int q = 0; q < 4; ++q) {
        const int e = blk * 4 + q;
        if (e >= per) break;
        // e = (((r * 2 + io) * C1 + c) * mh + i) * mw + j
        int rest = e;
        const int j = rest % mw; rest /= mw;
        const int i = rest % mh; rest /= mh;
        const int c = rest % C1; rest /= C1;
        const int io = rest & 1;
        const int r = rest >> 1;
        const size_t rule = size_t(s) * R + r;
        const size_t at = rule * pat + (size_t(c) * mh + i) * mw + j;
        const int8_t *src = io ? out_src : in_src;
        int8_t *dst = io ? out_dst : in_dst;
        int8_t v = src[at];
        if (i < shape[2 * rule] && j < shape[2 * rule + 1] && ((m.entry_channels >> c) & 1u) &&
            w[2 * q] < m.entry_p32)
            v = other_value(v, w[2 * q + 1] & 1u);
        dst[at] = v;
    }
}

__global__ void __launch_bounds__(256) mutate_rewards_kernel(const int32_t *src, int32_t *dst,
                                                             int S, int R, int64_t blocks_per,
                                                             MutateArgs m) {
    const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t >= int64_t(S) * blocks_per) return;
    const int s = int(t / blocks_per);
    const int64_t blk = t - int64_t(s) * blocks_per;
    uint32_t w[8];
    philox_words(m.seed, m.generation, uint64_t(s), 3, uint64_t(blk), w);
    const uint64_t span = uint64_t(int64_t(m.reward_hi) - int64_t(m.reward_lo) + 1);
    for (int q = 0; q < 4; ++q) {
        const int64_t r = blk * 4 + q;
        if (r >= R) break;
        const size_t at = size_t(s) * R + size_t(r);
        int32_t v = src[at];
        if (w[2 * q] < m.reward_p32)
            v = int32_t(int64_t(m.reward_lo) + int64_t(uint64_t(w[2 * q + 1]) % span));
        dst[at] = v;
    }
}

unsigned grid_for(int64_t threads) { return unsigned((threads + 255) / 256); }

}  // namespace

hipError_t launch_mutate_maps(const uint8_t *src, uint8_t *dst, int n, int C, int H, int W,
                              const MutateArgs &m, hipStream_t s) {
    const int per = C * H * W;                 // <= 31 * 64 * 64 in the batch API; any int here
    const int blocks_per = (per + 7) / 8;
    const int chunk = std::max(1, int((int64_t(1) << 30) / blocks_per));   // t fits 31 bits
    for (int k0 = 0; k0 < n; k0 += chunk) {
        const int nk = std::min(chunk, n - k0);
        const int64_t threads = int64_t(nk) * blocks_per;
        hipLaunchKernelGGL(mutate_maps_kernel, dim3(grid_for(threads)), dim3(256), 0, s, src, dst,
                           k0, nk, per, H * W, blocks_per, m);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_mutate_rules(int S, int R, int C, int mh, int mw, const int32_t *shape,
                               const int8_t *in_src, const int8_t *out_src,
                               const int32_t *reward_src, int8_t *in_dst, int8_t *out_dst,
                               int32_t *reward_dst, const MutateArgs &m, hipStream_t s) {
    if (int64_t(S) * R == 0) return hipSuccess;
    const int C1 = C + 1;
    const int per = R * 2 * C1 * mh * mw;     // <= 252 * 2 * 32 * 16 * 16
    const int eb = (per + 3) / 4;
    const int chunk = std::max(1, int((int64_t(1) << 30) / eb));
    for (int s0 = 0; s0 < S; s0 += chunk) {
        const int ns = std::min(chunk, S - s0);
        hipLaunchKernelGGL(mutate_entries_kernel, dim3(grid_for(int64_t(ns) * eb)), dim3(256), 0,
                           s, shape, in_src, out_src, in_dst, out_dst, s0, ns, R, C1, mh, mw, eb,
                           m);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t rb = (int64_t(R) + 3) / 4;
    hipLaunchKernelGGL(mutate_rewards_kernel, dim3(grid_for(int64_t(S) * rb)), dim3(256), 0, s,
                       reward_src, reward_dst, S, R, rb, m);
    return hipGetLastError();
}

}  // namespace av
