/* avo.c — CPU oracle for the Autoverse batched rule step (arXiv 2407.04221).
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: used only by the tests, the smoke check
 * and the benchmark's CPU baseline.  Plain, slow and literal on purpose; shares no code
 * with the GPU library.
 *
 * One step of one environment, in the paper's terms:
 *  1. The stored map D (C binary channels) is extended by a zero force plane F
 *     (Sec. 2.1: the player places invisible force tiles next to itself).
 *  2. The action (1 up, 2 right, 3 down, 4 left) puts a force tile on the on-map neighbour
 *     of every player cell in that direction; 0 (and >= 5) places none.
 *  3. The rule list is four built-in move rules (Sec. 2.1: the player moves onto an adjacent
 *     unobstructed cell holding force and consumes the force; Sec. 2.2.1: walls block it),
 *     then the environment's loaded rules in index order.
 *  4. Every rule is matched at every anchor (top-left corner) where its n x m patch lies on
 *     the map, all rules against the same extended map: rules are applied in parallel
 *     (Sec. 2.1.1).  A match needs every specified input entry to equal the map; this is
 *     the thresholded convolution of Sec. 2.1 (weights +1 for 1, -1 for must-be-0, 0 for
 *     don't care; threshold = number of 1 entries).
 *  5. Reward = sum over rules of the rule's reward times its number of matches
 *     (Sec. 2.2.1: a rule's reward is paid whenever it is applied).
 *  6. Each match votes the output kernel K_O = O - I onto the patch (Sec. 2.1, the
 *     transposed-convolution write), with don't-care read as: no vote where O is
 *     don't care, and the target value where only I is don't care.
 *  7. Every cell of every plane (F included) becomes 1 iff old value + votes >= 1, which
 *     keeps the multi-hot map binary (Sec. 2.2.1).
 *     In sequential mode (the paper's alternative "sequence of convolutions" reading),
 *     steps 4-7 run once per rule in list order instead: each rule is matched on the map
 *     the rules before it left, and its own votes are applied before the next rule.
 *     With rule application control (Sec. 2.1.1), a loaded rule's matches are first
 *     filtered: matches whose patch overlaps an applied match of an inhibiting earlier rule
 *     are dropped, and of the rest only the `limit` ones with the largest index-channel
 *     value are kept; rewards and votes use the kept matches.
 *  8. F is dropped.  The step counter advances; the episode is done when no player tile
 *     is left (a kill rule, Sec. 2.2.1) or the counter reaches the episode length.
 *     A done environment is reset to its initial map within the same step.
 */
#include "avo.h"

#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { CH_EMPTY = 0, CH_WALL = 1, CH_PLAYER = 2, CH_GOAL = 3 };

struct avo_batch {
    int B, H, W, C, max_rules, max_h, max_w, per_env, episode_len;
    int R;               /* loaded rules per set */
    int rule_mode;       /* 0 parallel, 1 sequential */
    int have_rules, have_maps;
    int32_t *shape;      /* [S][R][2] */
    int8_t *in_pat;      /* [S][R][C+1][max_h][max_w] */
    int8_t *out_pat;
    int32_t *reward;     /* [S][R] */
    uint8_t *maps;       /* [B][C][H][W] */
    uint8_t *init_maps;  /* [B][C][H][W] */
    int32_t *t;          /* [B] steps since the last reset */
    int32_t *limit;      /* [S][R] or NULL: matches applied per step, 0 = all */
    uint8_t *inhibit;    /* [S][R][R] or NULL: [q][r] = rule q inhibits rule r */
    int site_order;      /* 0 row-major, 1 random index channel */
    uint64_t seed;       /* key of the random index channel */
    uint64_t step_no;    /* batch steps since avo_reset */
};

/* A rule as the step uses it: patterns over C+1 channels, n x m, with its reward. */
typedef struct {
    int n, m;
    int reward;
    const int8_t *in;    /* [C+1][max_h][max_w] */
    const int8_t *out;
    int ph, pw;          /* row / column extent of the pattern arrays */
} rule_view;

static int pat_at(const int8_t *p, int ph, int pw, int c, int i, int j)
{
    return p[((size_t)c * ph + i) * pw + j];
}

/* Output-kernel entry: K_O = O - I where both are specified; with I don't care the vote
 * points at O; with O don't care there is no vote. */
static int kernel_out(int in, int out)
{
    if (out == -1) return 0;
    if (out == 1) return in == 1 ? 0 : 1;
    return in == 0 ? 0 : -1;  /* out == 0 */
}

int avo_create(int B, int H, int W, int C, int max_rules, int max_h, int max_w,
               int per_env, int episode_len, avo_batch **out)
{
    if (!out) return AVO_EINVAL;
    *out = NULL;
    if (B <= 0 || H <= 0 || W <= 0 || C < 4 || C > 31 || max_rules < 0 || max_h <= 0 ||
        max_w <= 0 || episode_len < 0 || (per_env != 0 && per_env != 1))
        return AVO_EINVAL;
    avo_batch *ab = (avo_batch *)calloc(1, sizeof(avo_batch));
    if (!ab) return AVO_ENOMEM;
    ab->B = B; ab->H = H; ab->W = W; ab->C = C;
    ab->max_rules = max_rules; ab->max_h = max_h; ab->max_w = max_w;
    ab->per_env = per_env; ab->episode_len = episode_len;
    size_t cells = (size_t)B * C * H * W;
    ab->maps = (uint8_t *)calloc(cells, 1);
    ab->init_maps = (uint8_t *)calloc(cells, 1);
    ab->t = (int32_t *)calloc((size_t)B, sizeof(int32_t));
    if (!ab->maps || !ab->init_maps || !ab->t) { avo_destroy(ab); return AVO_ENOMEM; }
    *out = ab;
    return AVO_OK;
}

int avo_load_rules(avo_batch *ab, int R, const int32_t *shape, const int8_t *in_pat,
                   const int8_t *out_pat, const int32_t *reward)
{
    if (!ab || R < 0 || R > ab->max_rules) return AVO_EINVAL;
    if (R > 0 && (!shape || !in_pat || !out_pat || !reward)) return AVO_EINVAL;
    int S = ab->per_env ? ab->B : 1;
    size_t pat = (size_t)(ab->C + 1) * ab->max_h * ab->max_w;
    for (int s = 0; s < S; s++) {
        long long worst = 0;
        for (int r = 0; r < R; r++) {
            int n = shape[((size_t)s * R + r) * 2 + 0];
            int m = shape[((size_t)s * R + r) * 2 + 1];
            if (n < 1 || m < 1 || n > ab->max_h || m > ab->max_w || n > ab->H || m > ab->W)
                return AVO_EINVAL;
            long long rw = reward[(size_t)s * R + r];
            worst += (rw < 0 ? -rw : rw) * (long long)(ab->H - n + 1) * (ab->W - m + 1);
            for (size_t e = 0; e < pat; e++) {
                int a = in_pat[((size_t)s * R + r) * pat + e];
                int b = out_pat[((size_t)s * R + r) * pat + e];
                if (a < -1 || a > 1 || b < -1 || b > 1) return AVO_EINVAL;
            }
        }
        if (worst >= AVO_REWARD_LIMIT) return AVO_EINVAL;
    }
    free(ab->shape); free(ab->in_pat); free(ab->out_pat); free(ab->reward);
    free(ab->limit); free(ab->inhibit);
    ab->shape = NULL; ab->in_pat = NULL; ab->out_pat = NULL; ab->reward = NULL;
    ab->limit = NULL; ab->inhibit = NULL;
    ab->site_order = 0; ab->seed = 0;
    ab->R = R;
    size_t nr = (size_t)S * R;
    if (nr > 0) {
        ab->shape = (int32_t *)malloc(nr * 2 * sizeof(int32_t));
        ab->in_pat = (int8_t *)malloc(nr * pat);
        ab->out_pat = (int8_t *)malloc(nr * pat);
        ab->reward = (int32_t *)malloc(nr * sizeof(int32_t));
        if (!ab->shape || !ab->in_pat || !ab->out_pat || !ab->reward) return AVO_ENOMEM;
        memcpy(ab->shape, shape, nr * 2 * sizeof(int32_t));
        memcpy(ab->in_pat, in_pat, nr * pat);
        memcpy(ab->out_pat, out_pat, nr * pat);
        memcpy(ab->reward, reward, nr * sizeof(int32_t));
    }
    ab->have_rules = 1;
    return AVO_OK;
}

int avo_reset(avo_batch *ab, const uint8_t *init_maps)
{
    if (!ab || !init_maps) return AVO_EINVAL;
    size_t cells = (size_t)ab->B * ab->C * ab->H * ab->W;
    for (size_t k = 0; k < cells; k++) {
        ab->init_maps[k] = init_maps[k] ? 1 : 0;
        ab->maps[k] = ab->init_maps[k];
    }
    memset(ab->t, 0, (size_t)ab->B * sizeof(int32_t));
    ab->step_no = 0;
    ab->have_maps = 1;
    return AVO_OK;
}

/* The four built-in move rules (Sec. 2.1 / Sec. 2.2.1), as 2x2 pattern arrays over C+1
 * channels with the anchor at the top-left.  Source cell: player 1 -> player 0.  Target
 * cell: force 1 and wall must-be-0 -> player 1, force 0. */
static void build_move_rules(int C, int8_t in[4][32][2][2], int8_t out[4][32][2][2],
                             int nm[4][2])
{
    /* (source, target) cell coordinates inside the pattern, and the pattern size */
    static const int src_tgt[4][4] = {
        /* right: source (0,0), target (0,1) */ {0, 0, 0, 1},
        /* left:  source (0,1), target (0,0) */ {0, 1, 0, 0},
        /* down:  source (0,0), target (1,0) */ {0, 0, 1, 0},
        /* up:    source (1,0), target (0,0) */ {1, 0, 0, 0},
    };
    static const int size[4][2] = {{1, 2}, {1, 2}, {2, 1}, {2, 1}};
    int F = C;
    for (int k = 0; k < 4; k++) {
        memset(in[k], -1, sizeof(in[k]));
        memset(out[k], -1, sizeof(out[k]));
        int sy = src_tgt[k][0], sx = src_tgt[k][1], ty = src_tgt[k][2], tx = src_tgt[k][3];
        in[k][CH_PLAYER][sy][sx] = 1;
        out[k][CH_PLAYER][sy][sx] = 0;
        in[k][F][ty][tx] = 1;
        in[k][CH_WALL][ty][tx] = 0;
        out[k][CH_PLAYER][ty][tx] = 1;
        out[k][F][ty][tx] = 0;
        nm[k][0] = size[k][0];
        nm[k][1] = size[k][1];
    }
}

static int rule_matches(const uint8_t *X, int H, int W, const rule_view *rv, int C1,
                        int ay, int ax)
{
    for (int c = 0; c < C1; c++)
        for (int i = 0; i < rv->n; i++)
            for (int j = 0; j < rv->m; j++) {
                int want = pat_at(rv->in, rv->ph, rv->pw, c, i, j);
                if (want == -1) continue;
                if (X[((size_t)c * H + ay + i) * W + ax + j] != want) return 0;
            }
    return 1;
}

/* Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds of two 64 x 64 -> 128-bit
 * multiplications with a Weyl-sequence key schedule. */
void avo_philox4x64(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4])
{
    uint64_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint64_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; round++) {
        unsigned __int128 p0 = (unsigned __int128)0xD2E7470EE14C6C93ULL * x0;
        unsigned __int128 p1 = (unsigned __int128)0xCA5A826395121157ULL * x2;
        uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0;
        uint64_t hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
        x0 = hi1 ^ x1 ^ k0;
        x1 = lo1;
        x2 = hi0 ^ x3 ^ k1;
        x3 = lo0;
        k0 += 0x9E3779B97F4A7C15ULL;
        k1 += 0xBB67AE8584CAA73BULL;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

uint32_t avo_random_word(uint64_t seed, uint64_t generation, uint64_t individual,
                         uint64_t stream, uint64_t word)
{
    uint64_t ctr[4] = {word / 8, generation, individual, stream};
    uint64_t key[2] = {seed, 0};
    uint64_t out[4];
    avo_philox4x64(ctr, key, out);
    int w = (int)(word % 8);
    return (uint32_t)(out[w / 2] >> (32 * (w % 2)));
}

uint32_t avo_site_key(int order, uint64_t seed, uint64_t n, int b, int pos)
{
    uint32_t rank = (uint32_t)(4095 - pos);
    if (order == 0) return rank;
    /* the site channel is stream 0 with the batch step number in the generation word */
    uint32_t u = avo_random_word(seed, n, (uint64_t)b, 0, (uint64_t)pos);
    return (u & 0xFFFFF000u) | rank;
}

/* Is the match of loaded rule r (set s) at (ay, ax), an n x m patch, inhibited: does its
 * patch overlap the patch of an applied match of some rule q < r that inhibits r?
 * applied[q] holds the applied anchors of loaded rule q in this step. */
static int inhibited(const avo_batch *ab, int s, int r, int n, int m, int ay, int ax,
                     const uint8_t *applied)
{
    const int H = ab->H, W = ab->W, R = ab->R;
    const size_t plane = (size_t)H * W;
    for (int q = 0; q < r; q++) {
        if (!ab->inhibit[((size_t)s * R + q) * R + r]) continue;
        int nq = ab->shape[((size_t)s * R + q) * 2 + 0];
        int mq = ab->shape[((size_t)s * R + q) * 2 + 1];
        /* patches [by, by+nq) x [bx, bx+mq) and [ay, ay+n) x [ax, ax+m) overlap */
        for (int by = 0; by + nq <= H; by++)
            for (int bx = 0; bx + mq <= W; bx++) {
                if (!applied[(size_t)q * plane + (size_t)by * W + bx]) continue;
                if (by < ay + n && ay < by + nq && bx < ax + m && ax < bx + mq) return 1;
            }
    }
    return 0;
}

static int cmp_desc_u32(const void *a, const void *b)
{
    uint32_t x = *(const uint32_t *)a, y = *(const uint32_t *)b;
    return x < y ? 1 : (x > y ? -1 : 0);
}

static void step_env(avo_batch *ab, int b, uint8_t action, float *reward_out,
                     uint8_t *done_out, uint8_t *X, int32_t *delta, uint8_t *applied,
                     uint32_t *keys)
{
    const int H = ab->H, W = ab->W, C = ab->C, C1 = C + 1, F = C;
    const size_t plane = (size_t)H * W;
    uint8_t *D = ab->maps + (size_t)b * C * plane;

    /* 1. extend the map by a zero force plane */
    memcpy(X, D, (size_t)C * plane);
    memset(X + (size_t)F * plane, 0, plane);

    /* 2. force tiles next to every player cell, in the action's direction */
    static const int dir[5][2] = {{0, 0}, {-1, 0}, {0, 1}, {1, 0}, {0, -1}};
    if (action >= 1 && action <= 4) {
        int dy = dir[action][0], dx = dir[action][1];
        for (int y = 0; y < H; y++)
            for (int x = 0; x < W; x++) {
                if (!X[(size_t)CH_PLAYER * plane + (size_t)y * W + x]) continue;
                int ty = y + dy, tx = x + dx;
                if (ty < 0 || ty >= H || tx < 0 || tx >= W) continue;
                X[(size_t)F * plane + (size_t)ty * W + tx] = 1;
            }
    }

    /* 3. the rule list: built-in moves, then the loaded set */
    int8_t mv_in[4][32][2][2], mv_out[4][32][2][2];
    int mv_nm[4][2];
    build_move_rules(C, mv_in, mv_out, mv_nm);
    int s = ab->per_env ? b : 0;
    int nrules = 4 + ab->R;
    size_t pat = (size_t)C1 * ab->max_h * ab->max_w;

    /* 4-6. match every rule at every valid anchor of the same map; sum rewards and votes */
    memset(delta, 0, (size_t)C1 * plane * sizeof(int32_t));
    long long rho = 0;
    for (int r = 0; r < nrules; r++) {
        rule_view rv;
        if (r < 4) {
            rv.n = mv_nm[r][0]; rv.m = mv_nm[r][1]; rv.reward = 0;
            rv.in = &mv_in[r][0][0][0]; rv.out = &mv_out[r][0][0][0];
            rv.ph = 2; rv.pw = 2;
        } else {
            size_t k = (size_t)s * ab->R + (r - 4);
            rv.n = ab->shape[k * 2 + 0]; rv.m = ab->shape[k * 2 + 1];
            rv.reward = ab->reward[k];
            rv.in = ab->in_pat + k * pat; rv.out = ab->out_pat + k * pat;
            rv.ph = ab->max_h; rv.pw = ab->max_w;
        }
        /* the rule's matches; with application control, filtered (Sec. 2.1.1) */
        const int loaded = r >= 4;
        uint8_t *A = applied + (size_t)(loaded ? r - 4 : ab->R) * plane;  /* moves: last slot */
        const int lim = (loaded && ab->limit) ? ab->limit[(size_t)s * ab->R + (r - 4)] : 0;
        int count = 0;
        memset(A, 0, plane);
        for (int ay = 0; ay + rv.n <= H; ay++)
            for (int ax = 0; ax + rv.m <= W; ax++) {
                int hit = rule_matches(X, H, W, &rv, C1, ay, ax);
                if (hit && loaded && ab->inhibit &&
                    inhibited(ab, s, r - 4, rv.n, rv.m, ay, ax, applied))
                    hit = 0;
                if (!hit) continue;
                A[(size_t)ay * W + ax] = 1;
                count++;
            }
        if (lim > 0 && count > lim) {
            /* keep the lim matches with the largest keys: find the lim-th largest key */
            int nk = 0;
            for (size_t p = 0; p < plane; p++)
                if (A[p]) keys[nk++] = avo_site_key(ab->site_order, ab->seed, ab->step_no, b, (int)p);
            qsort(keys, (size_t)nk, sizeof(uint32_t), cmp_desc_u32);
            uint32_t cut = keys[lim - 1];
            for (size_t p = 0; p < plane; p++)
                if (A[p] && avo_site_key(ab->site_order, ab->seed, ab->step_no, b, (int)p) < cut)
                    A[p] = 0;
        }
        /* 5-6. reward and votes of the applied matches */
        for (size_t p = 0; p < plane; p++) {
            if (!A[p]) continue;
            const int ay = (int)(p / W), ax = (int)(p % W);
            rho += rv.reward;
            for (int c = 0; c < C1; c++)
                for (int i = 0; i < rv.n; i++)
                    for (int j = 0; j < rv.m; j++) {
                        int k = kernel_out(pat_at(rv.in, rv.ph, rv.pw, c, i, j),
                                           pat_at(rv.out, rv.ph, rv.pw, c, i, j));
                        delta[(size_t)c * plane + (size_t)(ay + i) * W + ax + j] += k;
                    }
        }
        if (ab->rule_mode == 1) {   /* sequential: this rule's votes take effect now */
            for (size_t k = 0; k < (size_t)C1 * plane; k++) {
                X[k] = (X[k] + delta[k] >= 1) ? 1 : 0;
                delta[k] = 0;
            }
        }
    }

    /* 7. clamp old + votes to {0, 1} on every plane */
    for (size_t k = 0; k < (size_t)C1 * plane; k++)
        X[k] = (X[k] + delta[k] >= 1) ? 1 : 0;

    /* 8. drop the force plane, advance the counter, detect the end of the episode */
    memcpy(D, X, (size_t)C * plane);
    ab->t[b] += 1;
    int any_player = 0;
    for (size_t k = 0; k < plane; k++)
        if (D[(size_t)CH_PLAYER * plane + k]) { any_player = 1; break; }
    int done = !any_player || (ab->episode_len > 0 && ab->t[b] == ab->episode_len);
    if (done) {
        memcpy(D, ab->init_maps + (size_t)b * C * plane, (size_t)C * plane);
        ab->t[b] = 0;
    }
    reward_out[b] = (float)rho;
    done_out[b] = (uint8_t)done;
}

int avo_step(avo_batch *ab, const uint8_t *actions, float *rewards, uint8_t *done,
             int nthreads, int *used)
{
    if (!ab || !actions || !rewards || !done) return AVO_EINVAL;
    if (!ab->have_rules || !ab->have_maps) return AVO_ESTATE;
    if (nthreads < 1) nthreads = 1;
#ifndef _OPENMP
    nthreads = 1;
#endif
    /* per-thread scratch: the extended map, the vote sums, the applied anchors of every
     * loaded rule and the keys of one rule's matches */
    const size_t plane = (size_t)ab->H * ab->W;
    const size_t ext = (size_t)(ab->C + 1) * plane;
    const size_t app = (size_t)(ab->R + 1) * plane;
    uint8_t *X = (uint8_t *)malloc(ext * nthreads);
    int32_t *delta = (int32_t *)malloc(ext * nthreads * sizeof(int32_t));
    uint8_t *applied = (uint8_t *)malloc(app * nthreads);
    uint32_t *keys = (uint32_t *)malloc(plane * nthreads * sizeof(uint32_t));
    if (!X || !delta || !applied || !keys) {
        free(X); free(delta); free(applied); free(keys);
        return AVO_ENOMEM;
    }
    int got = 1;
#ifdef _OPENMP
#pragma omp parallel for num_threads(nthreads) schedule(static)
#endif
    for (int b = 0; b < ab->B; b++) {
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
        if (tid == 0) got = omp_get_num_threads();
#endif
        step_env(ab, b, actions[b], rewards, done, X + (size_t)tid * ext,
                 delta + (size_t)tid * ext, applied + (size_t)tid * app,
                 keys + (size_t)tid * plane);
    }
    ab->step_no += 1;
    free(X);
    free(delta);
    free(applied);
    free(keys);
    if (used) *used = got;
    return AVO_OK;
}

int avo_set_rule_mode(avo_batch *ab, int mode)
{
    if (!ab || (mode != 0 && mode != 1)) return AVO_EINVAL;
    ab->rule_mode = mode;
    return AVO_OK;
}

int avo_set_rule_control(avo_batch *ab, const int32_t *limit, const uint8_t *inhibit,
                         int order, uint64_t seed)
{
    if (!ab || (order != 0 && order != 1)) return AVO_EINVAL;
    if (!ab->have_rules) return AVO_ESTATE;
    const int R = ab->R;
    const size_t S = ab->per_env ? (size_t)ab->B : 1;
    if (limit)
        for (size_t k = 0; k < S * R; k++)
            if (limit[k] < 0) return AVO_EINVAL;
    if (inhibit)
        for (size_t s = 0; s < S; s++)
            for (int q = 0; q < R; q++)
                for (int r = 0; r <= q; r++)
                    if (inhibit[(s * R + q) * R + r]) return AVO_EINVAL;
    free(ab->limit); free(ab->inhibit);
    ab->limit = NULL; ab->inhibit = NULL;
    if (limit && R > 0) {
        ab->limit = (int32_t *)malloc(S * R * sizeof(int32_t));
        if (!ab->limit) return AVO_ENOMEM;
        memcpy(ab->limit, limit, S * R * sizeof(int32_t));
    }
    if (inhibit && R > 0) {
        ab->inhibit = (uint8_t *)malloc(S * R * R);
        if (!ab->inhibit) return AVO_ENOMEM;
        memcpy(ab->inhibit, inhibit, S * R * R);
    }
    ab->site_order = order;
    ab->seed = seed;
    return AVO_OK;
}

int avo_mutate_maps(const uint8_t *src, uint8_t *dst, int n, int C, int H, int W,
                    const avo_mutation *m)
{
    if (!src || !dst || !m || n < 0 || C < 1 || H < 1 || W < 1) return AVO_EINVAL;
    const size_t per = (size_t)C * H * W;
    for (int k = 0; k < n; k++)
        for (size_t e = 0; e < per; e++) {
            int c = (int)(e / ((size_t)H * W));
            int bit = src[(size_t)k * per + e] != 0;
            int flip = ((m->map_channels >> c) & 1) &&
                       avo_random_word(m->seed, m->generation, (uint64_t)k, 1, e) < m->map_flip_p32;
            dst[(size_t)k * per + e] = (uint8_t)(bit ^ flip);
        }
    return AVO_OK;
}

/* The value a changed entry takes: the lower or the higher of the two others. */
static int8_t other_value(int8_t old, int higher)
{
    int v = (old == -1 || old == 0) ? old : 1;
    int lo = v == -1 ? 0 : -1;          /* the two values of {-1, 0, 1} other than v */
    int hi = v == 1 ? 0 : 1;
    return (int8_t)(higher ? hi : lo);
}

int avo_mutate_rules(int S, int R, int C, int mh, int mw, const int32_t *shape,
                     const int8_t *in_src, const int8_t *out_src, const int32_t *reward_src,
                     int8_t *in_dst, int8_t *out_dst, int32_t *reward_dst,
                     const avo_mutation *m)
{
    if (!m || S < 0 || R < 0 || C < 1 || C > 31 || mh < 1 || mw < 1) return AVO_EINVAL;
    if (m->reward_lo > m->reward_hi) return AVO_EINVAL;
    if ((size_t)S * R > 0 && (!shape || !in_src || !out_src || !reward_src || !in_dst ||
                              !out_dst || !reward_dst))
        return AVO_EINVAL;
    const int C1 = C + 1;
    const size_t pat = (size_t)C1 * mh * mw;
    const uint64_t span = (uint64_t)((int64_t)m->reward_hi - (int64_t)m->reward_lo + 1);
    for (int s = 0; s < S; s++)
        for (int r = 0; r < R; r++) {
            const size_t k = (size_t)s * R + r;
            const int n = shape[k * 2 + 0], mm = shape[k * 2 + 1];
            for (int io = 0; io < 2; io++) {
                const int8_t *src = (io ? out_src : in_src) + k * pat;
                int8_t *dst = (io ? out_dst : in_dst) + k * pat;
                for (int c = 0; c < C1; c++)
                    for (int i = 0; i < mh; i++)
                        for (int j = 0; j < mw; j++) {
                            const size_t at = ((size_t)c * mh + i) * mw + j;
                            const uint64_t e = ((((uint64_t)r * 2 + io) * C1 + c) * mh + i) * mw + j;
                            int8_t v = src[at];
                            if (i < n && j < mm && ((m->entry_channels >> c) & 1) &&
                                avo_random_word(m->seed, m->generation, (uint64_t)s, 2, 2 * e) <
                                    m->entry_p32) {
                                uint32_t pick = avo_random_word(m->seed, m->generation,
                                                                (uint64_t)s, 2, 2 * e + 1);
                                v = other_value(v, (int)(pick & 1));
                            }
                            dst[at] = v;
                        }
            }
            int32_t rw = reward_src[k];
            if (avo_random_word(m->seed, m->generation, (uint64_t)s, 3, 2 * (uint64_t)r) <
                m->reward_p32) {
                uint32_t u = avo_random_word(m->seed, m->generation, (uint64_t)s, 3,
                                             2 * (uint64_t)r + 1);
                rw = (int32_t)((int64_t)m->reward_lo + (int64_t)(u % span));
            }
            reward_dst[k] = rw;
        }
    return AVO_OK;
}

int avo_get_maps(const avo_batch *ab, uint8_t *dst)
{
    if (!ab || !dst) return AVO_EINVAL;
    memcpy(dst, ab->maps, (size_t)ab->B * ab->C * ab->H * ab->W);
    return AVO_OK;
}

int avo_observe(const avo_batch *ab, int w, uint8_t *dst)
{
    if (!ab || !dst || w < 1) return AVO_EINVAL;
    const int H = ab->H, W = ab->W, C = ab->C;
    const size_t plane = (size_t)H * W;
    for (int b = 0; b < ab->B; b++) {
        const uint8_t *D = ab->maps + (size_t)b * C * plane;
        uint8_t *out = dst + (size_t)b * C * w * w;
        memset(out, 0, (size_t)C * w * w);
        int py = -1, px = -1;
        for (int y = 0; y < H && py < 0; y++)
            for (int x = 0; x < W; x++)
                if (D[(size_t)CH_PLAYER * plane + (size_t)y * W + x]) { py = y; px = x; break; }
        if (py < 0) continue;
        for (int c = 0; c < C; c++)
            for (int wy = 0; wy < w; wy++)
                for (int wx = 0; wx < w; wx++) {
                    int y = py - w / 2 + wy, x = px - w / 2 + wx;
                    if (y < 0 || y >= H || x < 0 || x >= W) continue;
                    out[((size_t)c * w + wy) * w + wx] = D[(size_t)c * plane + (size_t)y * W + x];
                }
    }
    return AVO_OK;
}

int avo_rule_features(const avo_batch *ab, uint8_t *dst)
{
    if (!ab || !dst) return AVO_EINVAL;
    if (!ab->have_rules) return AVO_ESTATE;
    const int S = ab->per_env ? ab->B : 1;
    const size_t pat = (size_t)(ab->C + 1) * ab->max_h * ab->max_w;
    for (size_t k = 0; k < (size_t)S * ab->R; k++)
        for (int io = 0; io < 2; io++) {
            const int8_t *src = (io ? ab->out_pat : ab->in_pat) + k * pat;
            uint8_t *spec = dst + ((k * 2 + io) * 2 + 0) * pat;
            uint8_t *val = dst + ((k * 2 + io) * 2 + 1) * pat;
            for (size_t e = 0; e < pat; e++) {
                spec[e] = src[e] != -1;
                val[e] = src[e] == 1;
            }
        }
    return AVO_OK;
}

int avo_get_counters(const avo_batch *ab, int32_t *dst)
{
    if (!ab || !dst) return AVO_EINVAL;
    memcpy(dst, ab->t, (size_t)ab->B * sizeof(int32_t));
    return AVO_OK;
}

int avo_set_counters(avo_batch *ab, const int32_t *src)
{
    if (!ab || !src) return AVO_EINVAL;
    for (int b = 0; b < ab->B; b++)
        if (src[b] < 0) return AVO_EINVAL;
    memcpy(ab->t, src, (size_t)ab->B * sizeof(int32_t));
    return AVO_OK;
}

void avo_destroy(avo_batch *ab)
{
    if (!ab) return;
    free(ab->shape); free(ab->in_pat); free(ab->out_pat); free(ab->reward);
    free(ab->maps); free(ab->init_maps); free(ab->t);
    free(ab->limit); free(ab->inhibit);
    free(ab);
}
