// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
// SC 2011): a counter-based generator, ten rounds of two 64 x 64 -> 128-bit products with a
// Weyl-sequence key schedule.  The library's random draws (the random site channel of rule
// application control, the mutation operators) are 32-bit words of its output: word w of a
// stream is half (w % 2, low half first) of 64-bit output word (w % 8) / 2 of the block at
// counter (w / 8, generation, individual, stream), key (seed, 0).
//
// Plain types only, so that the lane16 programs compiled at run time can include this text.
#pragma once

#ifndef __HIPCC_RTC__
#include <hip/hip_runtime.h>
#endif

namespace av {

typedef unsigned long long philox_u64;

// Full 64 x 64 -> 128-bit product from four 32 x 32 + 64 multiply-adds (one
// v_mad_u64_u32 each); no partial sum overflows: (2^32 - 1)^2 + 2 (2^32 - 1) = 2^64 - 1.
__device__ inline void mul64x64(philox_u64 a, philox_u64 x, philox_u64 &lo, philox_u64 &hi) {
    const unsigned int al = (unsigned int)a, ah = (unsigned int)(a >> 32);
    const unsigned int xl = (unsigned int)x, xh = (unsigned int)(x >> 32);
    const philox_u64 t0 = (philox_u64)al * xl;
    const philox_u64 t1 = (philox_u64)al * xh + (t0 >> 32);
    const philox_u64 t2 = (philox_u64)ah * xl + (unsigned int)t1;
    hi = (philox_u64)ah * xh + (t1 >> 32) + (t2 >> 32);
    lo = (t2 << 32) | (unsigned int)t0;
}

__device__ inline void philox4x64_10(philox_u64 x[4], philox_u64 k0, philox_u64 k1) {
    for (int round = 0; round < 10; ++round) {
        philox_u64 lo0, hi0, lo1, hi1;
        mul64x64(0xD2E7470EE14C6C93ull, x[0], lo0, hi0);
        mul64x64(0xCA5A826395121157ull, x[2], lo1, hi1);
        const philox_u64 y0 = hi1 ^ x[1] ^ k0, y2 = hi0 ^ x[3] ^ k1;
        x[0] = y0; x[1] = lo1; x[2] = y2; x[3] = lo0;
        k0 += 0x9E3779B97F4A7C15ull;
        k1 += 0xBB67AE8584CAA73Bull;
    }
}

// The eight 32-bit words of block `blk` of a stream.
__device__ inline void philox_words(philox_u64 seed, philox_u64 generation, philox_u64 individual,
                                    philox_u64 stream, philox_u64 blk, unsigned int w[8]) {
    philox_u64 x[4] = {blk, generation, individual, stream};
    philox4x64_10(x, seed, 0);
    for (int j = 0; j < 4; ++j) {
        w[2 * j] = (unsigned int)x[j];
        w[2 * j + 1] = (unsigned int)(x[j] >> 32);
    }
}

}  // namespace av
