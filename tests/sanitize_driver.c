/* Drives every entry point of the CPU oracle (oracle/avo.c) on seeded random inputs for a
 * build with AddressSanitizer and UndefinedBehaviorSanitizer (tests/test_oracle_sanitizers.py
 * compiles and runs it; test infrastructure only).  Every buffer is allocated at exactly the
 * size the API documents, so an access past the end of one is reported.  Returns 0 when every
 * call returned what it should; the sanitizers abort the process on any finding. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "avo.h"

static uint64_t g_state = 0x9E3779B97F4A7C15ull;

static uint32_t rnd(void) {            /* xorshift64* */
    g_state ^= g_state >> 12;
    g_state ^= g_state << 25;
    g_state ^= g_state >> 27;
    return (uint32_t)((g_state * 0x2545F4914F6CDD1Dull) >> 32);
}
static int rnd_in(int lo, int hi) { return lo + (int)(rnd() % (uint32_t)(hi - lo + 1)); }

static int g_fail = 0;
#define EXPECT(cond)                                                            \
    do {                                                                        \
        if (!(cond)) {                                                          \
            fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
            g_fail = 1;                                                         \
        }                                                                       \
    } while (0)

typedef struct {
    int B, H, W, C, R, mh, mw, per_env, L, T;
} Case;

static void run_case(const Case *k) {
    const int S = k->per_env ? k->B : 1, C1 = k->C + 1;
    const size_t pat = (size_t)C1 * k->mh * k->mw;
    const size_t cells = (size_t)k->B * k->C * k->H * k->W;
    avo_batch *ab = NULL;
    EXPECT(avo_create(k->B, k->H, k->W, k->C, k->R, k->mh, k->mw, k->per_env, k->L, &ab) == AVO_OK);
    if (!ab) return;

    int32_t *shape = malloc(sizeof(int32_t) * 2 * (size_t)S * k->R + 1);
    int8_t *in = malloc(pat * (size_t)S * k->R + 1), *out = malloc(pat * (size_t)S * k->R + 1);
    int32_t *reward = malloc(sizeof(int32_t) * (size_t)S * k->R + 1);
    for (int i = 0; i < S * k->R; ++i) {
        shape[2 * i] = rnd_in(1, k->mh < k->H ? k->mh : k->H);
        shape[2 * i + 1] = rnd_in(1, k->mw < k->W ? k->mw : k->W);
        reward[i] = rnd_in(-1, 1);
    }
    for (size_t e = 0; e < pat * (size_t)S * k->R; ++e) {
        /* mostly don't care, so that rules fire and votes of both signs overlap */
        in[e] = (int8_t)(rnd() % 4 ? -1 : rnd_in(0, 1));
        out[e] = (int8_t)(rnd() % 3 ? -1 : rnd_in(0, 1));
    }
    uint8_t *maps = malloc(cells), *acts = malloc((size_t)k->B), *done = malloc((size_t)k->B);
    float *rew = malloc(sizeof(float) * (size_t)k->B);
    for (size_t e = 0; e < cells; ++e) maps[e] = (uint8_t)(rnd() % 3 == 0);
    for (int b = 0; b < k->B; ++b)      /* one player in every map */
        maps[(((size_t)b * k->C + 2) * k->H + rnd_in(0, k->H - 1)) * k->W + rnd_in(0, k->W - 1)] = 1;

    /* calls out of order and bad arguments */
    EXPECT(avo_step(ab, acts, rew, done, 1, NULL) == AVO_ESTATE);
    EXPECT(avo_set_rule_control(ab, NULL, NULL, 0, 0) == AVO_ESTATE);
    EXPECT(avo_load_rules(ab, k->R + 1, shape, in, out, reward) == AVO_EINVAL);
    if (k->R > 0) {
        const int8_t keep = in[0];
        in[0] = 2;
        EXPECT(avo_load_rules(ab, k->R, shape, in, out, reward) == AVO_EINVAL);
        in[0] = keep;
    }
    EXPECT(avo_load_rules(ab, k->R, shape, in, out, reward) == AVO_OK);
    EXPECT(avo_reset(ab, maps) == AVO_OK);
    EXPECT(avo_set_rule_mode(ab, 2) == AVO_EINVAL);

    int32_t *limit = malloc(sizeof(int32_t) * (size_t)S * k->R + 1);
    uint8_t *inhibit = calloc((size_t)S * k->R * k->R + 1, 1);
    for (int i = 0; i < S * k->R; ++i) limit[i] = rnd_in(0, 3);
    for (int s = 0; s < S; ++s)
        for (int q = 0; q < k->R; ++q)
            for (int r = q + 1; r < k->R; ++r)
                inhibit[((size_t)s * k->R + q) * k->R + r] = (uint8_t)(rnd() % 4 == 0);

    const int w = rnd_in(1, 2 * k->H + 3);
    uint8_t *obs = malloc((size_t)k->B * k->C * w * w);
    uint8_t *feat = malloc(pat * (size_t)S * k->R * 4 + 1);
    int32_t *ctr = malloc(sizeof(int32_t) * (size_t)k->B);
    for (int t = 0; t < k->T; ++t) {
        if (t == k->T / 3) EXPECT(avo_set_rule_mode(ab, 1) == AVO_OK);
        if (t == k->T / 2) EXPECT(avo_set_rule_control(ab, limit, inhibit, t & 1, 77) == AVO_OK);
        for (int b = 0; b < k->B; ++b) acts[b] = (uint8_t)rnd_in(0, 7);
        int used = 0;
        EXPECT(avo_step(ab, acts, rew, done, 1 + (t & 3), &used) == AVO_OK);
        for (int b = 0; b < k->B; ++b) EXPECT(done[b] <= 1);
        EXPECT(avo_observe(ab, w, obs) == AVO_OK);
        EXPECT(avo_get_maps(ab, maps) == AVO_OK);
        EXPECT(avo_get_counters(ab, ctr) == AVO_OK);
    }
    EXPECT(avo_rule_features(ab, feat) == AVO_OK);
    for (int b = 0; b < k->B; ++b) ctr[b] = b % 3;
    EXPECT(avo_set_counters(ab, ctr) == AVO_OK);
    ctr[0] = -1;
    EXPECT(avo_set_counters(ab, ctr) == AVO_EINVAL);

    /* mutation operators, in place and out of place */
    avo_mutation m = {12345, 3, 1u << 28, 0xFFFFFFFFu, 1u << 29, 0xFFFFFFFFu, 1u << 30, -2, 2};
    uint8_t *maps2 = malloc(cells);
    EXPECT(avo_mutate_maps(maps, maps2, k->B, k->C, k->H, k->W, &m) == AVO_OK);
    EXPECT(avo_mutate_maps(maps2, maps2, k->B, k->C, k->H, k->W, &m) == AVO_OK);
    EXPECT(avo_mutate_rules(S, k->R, k->C, k->mh, k->mw, shape, in, out, reward, in, out, reward,
                            &m) == AVO_OK);
    m.reward_lo = 3;
    EXPECT(avo_mutate_rules(S, k->R, k->C, k->mh, k->mw, shape, in, out, reward, in, out, reward,
                            &m) == AVO_EINVAL);

    avo_destroy(ab);
    free(shape); free(in); free(out); free(reward); free(maps); free(maps2); free(acts);
    free(done); free(rew); free(limit); free(inhibit); free(obs); free(feat); free(ctr);
}

int main(void) {
    avo_batch *ab = NULL;
    EXPECT(avo_create(0, 4, 4, 4, 1, 1, 1, 0, 0, &ab) == AVO_EINVAL);
    EXPECT(avo_create(2, 4, 4, 3, 1, 1, 1, 0, 0, &ab) == AVO_EINVAL);
    EXPECT(avo_create(2, 4, 4, 32, 1, 1, 1, 0, 0, &ab) == AVO_EINVAL);
    EXPECT(avo_create(2, 4, 4, 4, 1, 1, 1, 2, 0, &ab) == AVO_EINVAL);
    EXPECT(ab == NULL);
    const Case cases[] = {
        {5, 7, 9, 4, 3, 3, 3, 0, 4, 12},      /* shared rules, short episodes */
        {4, 6, 5, 6, 4, 3, 2, 1, 0, 10},      /* per-environment rules */
        {3, 1, 16, 5, 2, 1, 4, 0, 3, 8},      /* one-row maps */
        {3, 16, 1, 5, 2, 4, 1, 1, 3, 8},      /* one-column maps */
        {2, 8, 8, 4, 2, 8, 8, 0, 5, 6},       /* patterns as large as the map */
        {2, 12, 64, 31, 3, 2, 5, 0, 4, 4},    /* the widest map, the most channels */
        {3, 5, 5, 4, 0, 1, 1, 0, 2, 6},       /* no loaded rules */
    };
    for (size_t i = 0; i < sizeof cases / sizeof cases[0]; ++i) run_case(&cases[i]);
    if (g_fail) return 1;
    printf("sanitize driver: all calls behaved\n");
    return 0;
}
