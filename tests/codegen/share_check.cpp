// Runs an emitted count function (share_emit.cpp's output, included as counts.inc) on random
// words and compares every bit with a direct count of the list's terms.
#include <cstdint>
#include <cstdio>
#include <random>

typedef uint32_t u32;
// v_bitop3_b32: bit i of the result is bit (4 a_i + 2 b_i + c_i) of the table
static u32 bitop3(u32 a, u32 b, u32 c, unsigned t) {
    u32 r = 0;
    for (int i = 0; i < 32; ++i) {
        const unsigned k = (((a >> i) & 1u) << 2) | (((b >> i) & 1u) << 1) | ((c >> i) & 1u);
        r |= ((t >> k) & 1u) << i;
    }
    return r;
}
#define __builtin_amdgcn_bitop3_b32(a, b, c, t) bitop3((a), (b), (c), (t))
#include "counts.inc"

int main() {
    std::mt19937 rng(7);
    u32 x[NIN], out[NOUT];
    for (int rep = 0; rep < 200; ++rep) {
        for (int i = 0; i < NIN; ++i) {
            // sparse, dense and even words
            const int kind = rng() % 3;
            u32 w = rng();
            if (kind == 0) w &= rng() & rng();
            if (kind == 1) w |= rng() | rng();
            x[i] = w;
        }
        counts(x, out);
        for (int l = 0; l < NOUT; ++l)
            for (int bit = 0; bit < 32; ++bit) {
                long n = 0;
                for (const int *t = kTerms[l]; *t; ++t) {
                    const int idx = (*t > 0 ? *t : -*t) - 1;
                    const u32 v = (x[idx] >> bit) & 1u;
                    n += *t > 0 ? v : 1u - v;
                }
                const u32 want = n >= kK[l] ? 1u : 0u;
                if (((out[l] >> bit) & 1u) != want) {
                    std::printf("mismatch: list %d bit %d count %ld K %ld\n", l, bit, n, kK[l]);
                    return 1;
                }
            }
    }
    std::printf("ok\n");
    return 0;
}
