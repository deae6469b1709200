// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
// SC 2011): a counter-based generator, ten rounds of two 64 x 64 -> 128-bit products with a
// Weyl-sequence key schedule.  The library's random draws (the random site channel of rule
// application control, the mutation operators) are 32-bit words of its output: word w of a
// stream is half (w % 2, low half first) of 64-bit output word (w % 8) / 2 of the block at
// counter (w / 8, generation, individual, stream), key (seed, 0).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace av {

// Full 64 x 64 -> 128-bit product from four 32 x 32 + 64 multiply-adds (one
// v_mad_u64_u32 each); no partial sum overflows: (2^32 - 1)^2 + 2 (2^32 - 1) = 2^64 - 1.
__device__ inline void mul64x64(uint64_t a, uint64_t x, uint64_t &lo, uint64_t &hi) {
    const uint32_t al = uint32_t(a), ah = uint32_t(a >> 32);
    const uint32_t xl = uint32_t(x), xh = uint32_t(x >> 32);
    const uint64_t t0 = uint64_t(al) * xl;
    const uint64_t t1 = uint64_t(al) * xh + (t0 >> 32);
    const uint64_t t2 = uint64_t(ah) * xl + uint32_t(t1);
    hi = uint64_t(ah) * xh + (t1 >> 32) + (t2 >> 32);
    lo = (t2 << 32) | uint32_t(t0);
}

__device__ inline void philox4x64_10(uint64_t x[4], uint64_t k0, uint64_t k1) {
    for (int round = 0; round < 10; ++round) {
        uint64_t lo0, hi0, lo1, hi1;
        mul64x64(0xD2E7470EE14C6C93ull, x[0], lo0, hi0);
        mul64x64(0xCA5A826395121157ull, x[2], lo1, hi1);
        const uint64_t y0 = hi1 ^ x[1] ^ k0, y2 = hi0 ^ x[3] ^ k1;
        x[0] = y0; x[1] = lo1; x[2] = y2; x[3] = lo0;
        k0 += 0x9E3779B97F4A7C15ull;
        k1 += 0xBB67AE8584CAA73Bull;
    }
}

// The eight 32-bit words of block `blk` of a stream.
__device__ inline void philox_words(uint64_t seed, uint64_t generation, uint64_t individual,
                                    uint64_t stream, uint64_t blk, uint32_t w[8]) {
    uint64_t x[4] = {blk, generation, individual, stream};
    philox4x64_10(x, seed, 0);
    for (int j = 0; j < 4; ++j) {
        w[2 * j] = uint32_t(x[j]);
        w[2 * j + 1] = uint32_t(x[j] >> 32);
    }
}

}  // namespace av
