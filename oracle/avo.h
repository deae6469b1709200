/* avo.h — CPU oracle for the Autoverse batched rule step (arXiv 2407.04221).
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test-suite, the smoke check and
 * the benchmark's CPU-baseline leg call this code.  It shares no source with the GPU
 * library; both are fed the same seeded arrays.
 *
 * The oracle is the plain definition of one environment step written out with int8 loops
 * over maps, rules, anchors and pattern entries (paper Sec. 2.1, the patch-replacement
 * equation generalised to many matches by the convolution / transposed-convolution pair,
 * Sec. 2.1.1 for parallel rule application, Sec. 2.2.1 for force-tile moves, rewards and
 * kill rules).  All arrays are host memory.
 *
 * Layouts (all C-contiguous):
 *   maps, init_maps  uint8 [B][C][H][W], values 0/1
 *   shape            int32 [S][R][2]  (rows n, cols m) of each rule
 *   in_pat, out_pat  int8  [S][R][C+1][max_h][max_w]; 1, 0, or -1 = don't care.
 *                    Channel C is the force plane.  Entries outside n x m are ignored.
 *   reward           int32 [S][R]
 *   actions          uint8 [B]  0 none, 1 up, 2 right, 3 down, 4 left; >= 5 acts as 0
 *   rewards          float [B], done uint8 [B]
 *   S = B when per_env is set, else 1.
 */
#ifndef AVO_H
#define AVO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { AVO_OK = 0, AVO_EINVAL = 1, AVO_ENOMEM = 2, AVO_ESTATE = 4 };

/* Largest |sum of rewards| one step may produce, so that the float output is exact. */
#define AVO_REWARD_LIMIT (1 << 24)

typedef struct avo_batch avo_batch;

int  avo_create(int B, int H, int W, int C, int max_rules, int max_h, int max_w,
                int per_env, int episode_len, avo_batch **out);
int  avo_load_rules(avo_batch *ab, int R, const int32_t *shape, const int8_t *in_pat,
                    const int8_t *out_pat, const int32_t *reward);
int  avo_reset(avo_batch *ab, const uint8_t *init_maps);
/* One step of every environment.  nthreads > 1 splits the environments over OpenMP
 * threads (they are independent); returns the thread count used through *used. */
int  avo_step(avo_batch *ab, const uint8_t *actions, float *rewards, uint8_t *done,
              int nthreads, int *used);
/* Rule order within a step: 0 = parallel (every rule matches the same map and all votes
 * are summed once, Sec. 2.1.1; the default), 1 = sequential (rules apply one after another
 * in list order, each matching the map the previous ones left; a rule's own matches are
 * applied together). */
int  avo_set_rule_mode(avo_batch *ab, int mode);
/* Rule application control (paper Sec. 2.1.1: rules may be made to apply only once or a
 * fixed number of times, in an ordered or a random order, by taking the maximum of an extra
 * channel of index values; masks can make some rules inhibit others).  Applies to the
 * loaded rules only (never to the four moves) and is cleared by avo_load_rules.
 *   limit    int32 [S][R] or NULL: at most limit matches of the rule apply per step;
 *            0 = every match applies.  Negative values are rejected.
 *   inhibit  uint8 [S][R][R] or NULL: inhibit[s][q][r] != 0 means a match of rule r is
 *            dropped when its patch overlaps the patch of an applied match of rule q in the
 *            same step.  Only q < r is allowed (rule index is priority).
 *   order    0: the kept matches are the first ones in row-major anchor order;
 *            1: they are the ones with the largest random index value (avo_site_key).
 *   seed     key of the random index channel.
 * Per rule and step: match, drop inhibited matches, keep the `limit` matches with the
 * largest keys, then pay rewards and vote with the kept ones. */
int  avo_set_rule_control(avo_batch *ab, const int32_t *limit, const uint8_t *inhibit,
                          int order, uint64_t seed);
/* The index-channel value of anchor (y, x) of environment b at batch step number n (steps
 * since avo_reset, all environments counted together): with pos = y * W + x, order 0 gives
 * 4095 - pos; order 1 gives the high 20 bits of a Philox4x64-10 word (Salmon et al. 2011;
 * counter (pos / 8, n, b, 0), key (seed, 0), 32-bit word pos % 8 of the output, low half of
 * each 64-bit word first) above 4095 - pos, so that keys never tie. */
uint32_t avo_site_key(int order, uint64_t seed, uint64_t n, int b, int pos);
/* Philox4x64-10 block function, exported so that tests can pin it. */
void avo_philox4x64(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]);
/* Mutation operators (paper Sec. 2.2.1 and the Fig. 2b caption: environments are mutated
 * by flipping bits of the initial multi-hot map, by changing entries of the rules' input
 * and output patterns, and by changing the rules' rewards).  Every random draw is a 32-bit
 * word of Philox4x64-10 (avo_random_word) with key (seed, 0) and counter
 * (word / 8, generation, individual, stream); stream 1 = map bits, 2 = pattern entries,
 * 3 = rewards.  Probabilities are 32-bit thresholds: an event with threshold p happens iff
 * its word is < p (probability p / 2^32). */
typedef struct {
    uint64_t seed, generation;
    uint32_t map_flip_p32;     /* per map bit */
    uint32_t map_channels;     /* bit c set: channel c of the map may flip */
    uint32_t entry_p32;        /* per pattern entry inside the rule's n x m */
    uint32_t entry_channels;   /* bit c set: entries of channel c (C = force) may change */
    uint32_t reward_p32;       /* per rule */
    int32_t reward_lo, reward_hi;
} avo_mutation;

/* 32-bit word `word` (pos % 8 of the block pos / 8, low half of each 64-bit word first). */
uint32_t avo_random_word(uint64_t seed, uint64_t generation, uint64_t individual,
                         uint64_t stream, uint64_t word);
/* Maps uint8 [n][C][H][W] (nonzero = tile): bit e = (c * H + y) * W + x of individual k
 * flips iff channel c is in map_channels and word e of stream 1 is < map_flip_p32.
 * dst holds 0/1; dst may equal src. */
int  avo_mutate_maps(const uint8_t *src, uint8_t *dst, int n, int C, int H, int W,
                     const avo_mutation *m);
/* Rules in the av_load_rules layout: shape [S][R][2], patterns [S][R][C+1][mh][mw],
 * rewards [S][R]; individual = set s.  Entry e = (((r * 2 + io) * (C+1) + c) * mh + i) * mw + j
 * (io 0 = input, 1 = output) with i < n, j < m of its rule and channel c in entry_channels
 * changes iff word 2e of stream 2 is < entry_p32; it then takes the lower (word 2e + 1 even)
 * or higher (odd) of the two values of {-1, 0, 1} other than its own (a value outside the
 * set counts as 1).  Reward r is redrawn iff word 2r of stream 3 is < reward_p32, to
 * reward_lo + (word 2r + 1) mod (reward_hi - reward_lo + 1).  Destinations may equal the
 * sources.  AVO_EINVAL if reward_lo > reward_hi. */
int  avo_mutate_rules(int S, int R, int C, int mh, int mw, const int32_t *shape,
                      const int8_t *in_src, const int8_t *out_src, const int32_t *reward_src,
                      int8_t *in_dst, int8_t *out_dst, int32_t *reward_dst,
                      const avo_mutation *m);
int  avo_get_maps(const avo_batch *ab, uint8_t *dst);
/* Player-centred observation of the current maps (paper Sec. 2.2.2: a local patch of tiles
 * around the player's position; Table 1 uses windows of 5, 10, 20 and 31 cells).
 * dst uint8 [B][C][w][w]: window cell (wy, wx) shows map cell (py - w/2 + wy, px - w/2 + wx),
 * with (py, px) the environment's first player cell in row-major order and w/2 rounded
 * down; cells off the map, and every cell when there is no player, are 0. */
int  avo_observe(const avo_batch *ab, int w, uint8_t *dst);
/* The loaded rules as binary features (paper Sec. 2.2.2: the observation also holds a binary
 * representation of the environment's rules).  dst uint8 [S][R][2][2][C+1][max_h][max_w]:
 * [.][.][0 = input, 1 = output][0 = entry specified, 1 = entry value (0 when unspecified)]. */
int  avo_rule_features(const avo_batch *ab, uint8_t *dst);
int  avo_get_counters(const avo_batch *ab, int32_t *dst);
/* Set every environment's step counter (t[b] >= 0), e.g. to a search node's depth. */
int  avo_set_counters(avo_batch *ab, const int32_t *src);
void avo_destroy(avo_batch *ab);

#ifdef __cplusplus
}
#endif
#endif
