/* autoverse.h — C ABI of libautoverse.so: the batched environment step of Autoverse
 * (Earle & Togelius, "Autoverse: an Evolvable Game Language for Learning Robust Embodied
 * Agents", arXiv 2407.04221) on one AMD Instinct MI355X (gfx950).
 *
 * What one step computes, for every environment independently (paper Sec. 2.1, Sec. 2.1.1,
 * Sec. 2.2.1):
 *   - the map is C binary channels ("tiles"), multi-hot per cell; channel 0 empty, 1 wall,
 *     2 player, 3 goal/food, 4.. extra tile types;
 *   - the action (0 none, 1 up, 2 right, 3 down, 4 left; larger values act as 0) places a
 *     transient force tile on the on-map neighbour of every player cell in that direction;
 *     the force plane is channel C while the step runs and is never stored;
 *   - four built-in move rules (player next to force on a wall-free cell moves there and
 *     consumes the force) and the loaded rules are matched, all against the same map
 *     (rules apply in parallel, Sec. 2.1.1), at every anchor where the pattern lies wholly
 *     on the map; a match needs every specified input entry to hold (the thresholded
 *     convolution of Sec. 2.1);
 *   - the reward is the sum over rules of the rule's reward times its number of matches;
 *   - every match votes K_O = O - I onto its patch (the transposed convolution of
 *     Sec. 2.1; an unspecified output entry votes nothing, an unspecified input entry
 *     votes toward the output); a cell-channel becomes 1 iff old value + votes >= 1;
 *   - the episode is done when no player tile is left (a kill rule, Sec. 2.2.1) or the step
 *     counter reaches max_episode_steps; a done environment is reset to its initial map
 *     within the same step, and that step's reward and done flag are still reported.
 *
 * Status codes only: no exception crosses this boundary.  Errors in arguments are found on
 * the host before any launch; device failures return AV_EDEVICE.  av_last_error() gives a
 * thread-local message for the last failing call on the calling thread.
 *
 * Memory: the library allocates and owns all persistent device state (packed maps,
 * initial maps, step counters, compiled rules).  The caller owns actions, rewards, done
 * and dst buffers: device pointers on the batch's device (for example torch tensors'
 * data_ptr()).  Host pointers appear only in av_load_rules, av_get_state, av_set_state.
 *
 * Ordering: all device work is issued on the batch's stream.  av_step and av_step_n never
 * synchronise; av_load_rules, av_reset, av_get_state, av_set_state and av_destroy_batch
 * may.  Calls on one batch must not overlap (one batch is not thread-safe); different
 * batches are independent.
 */
#ifndef AUTOVERSE_H
#define AUTOVERSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct av_batch_s *av_batch_t;

typedef enum {
    AV_OK = 0,
    AV_EINVAL = 1,   /* bad argument: NULL pointer, size out of range, bad pattern value */
    AV_ENOMEM = 2,   /* host or device allocation failed */
    AV_EDEVICE = 3,  /* a HIP call failed; av_last_error() names it */
    AV_ESTATE = 4    /* call out of order, e.g. av_step before av_load_rules and av_reset */
} av_status;

/* Kernel family used by av_step / av_step_n.  AUTO picks lane16 when eligible; else, for
 * per-environment rule sets, group when eligible, else wave when its LDS working set (C + 1
 * padded planes, one match plane per rule, two vote accumulators per plane) fits in 64 KiB;
 * else rows when eligible; else wave when it fits; else generic.  With rule application
 * control (av_set_rule_control) a batch created with AUTO runs lane16, or wave when the control
 * scratch fits its LDS, or generic. */
typedef enum {
    AV_ENGINE_AUTO = 0,
    AV_ENGINE_GENERIC = 1,  /* any size within the limits below; maps staged in LDS */
    AV_ENGINE_LANE16 = 2,   /* maps of at most 16 x 16 and one shared rule set: one map
                               row per lane, two maps per 32-bit lane word, rows shifted
                               across lanes with DPP, the rule set compiled into the kernel */
    AV_ENGINE_WAVE = 3,     /* one environment per workgroup, map rows in LDS; 4 to 64
                               groups of lanes (as many as the batch's size leaves room for)
                               match that many of its rules at once */
    AV_ENGINE_ROWS = 4,     /* one environment per 64-lane wave, map row y in lane y,
                               planes in the workgroup's LDS; one lane per rule tests every
                               rule's rarest entries at once, so only rules that can match
                               are visited.  On maps above 32 rows, in parallel rule order,
                               with 4 B waves within the device's wave slots, three more
                               waves per environment share the probe and the matching.
                               Needs R + 4 <= 64 and, within 64 KiB of LDS, (3 C + 4) planes
                               of H + 16 rows plus R + 4 match planes of H + 32 rows (4 bytes
                               per row for W <= 32, else 8), 36 bytes per rule and 96 more;
                               no rule application control */
    AV_ENGINE_GROUP = 5     /* one environment per 64-lane wave, no barriers: 4 groups of 16
                               lanes, lane y of each owning map row y (and row y + 16 on maps
                               of 17 to 32 rows), group g matching rules g, g + 4, ...; input
                               entries are merged per pattern row, every rule's first four
                               merged entries are tested in one round of LDS reads, and only
                               rules that pass somewhere read the rest.  After launches of 64 steps or more it measures each
                               environment's cycles and deals environments to workgroups so that
                               the slowest ones do not share a SIMD (results never depend on
                               the order; not while the stream is captured).  Needs parallel
                               rule order, H, W <= 32,
                               (max_rules + 4) x max_pat_h x max_pat_w <= 254, at most 8
                               channels per lane group and, within 64 KiB of LDS, C + 1 planes
                               and R + 4 match planes of HR + max_pat_h - 1 rows (rounded up to
                               4), 3 C rows of HR, 12 words per rule plus 12, and C (R + 6)
                               words, 4 bytes each (HR = 16, or 32 on maps of 17 to 32 rows);
                               no rule application control */
} av_engine;

/* Order in which the rules of one step are applied. */
typedef enum {
    AV_RULES_PARALLEL = 0,    /* every rule matches the same map; all votes summed once
                                 (paper Sec. 2.1.1; the default) */
    AV_RULES_SEQUENTIAL = 1   /* rules apply one after another in list order (the four moves,
                                 then the loaded rules by index); each matches the map the
                                 rules before it left, force plane included; all matches of
                                 one rule apply together (the "sequence of convolutions"
                                 reading of the Fig. 2a caption) */
} av_rule_mode;

typedef struct {
    int32_t num_envs;           /* B >= 1 */
    int32_t height, width;      /* H, W in [1, 64] */
    int32_t channels;           /* C in [4, 31]; patterns span C + 1 channels */
    int32_t max_rules;          /* most rules one av_load_rules may load, in [0, 252] */
    int32_t max_pat_h, max_pat_w; /* pattern array extent, each in [1, 16] */
    int32_t per_env_rules;      /* 0: one rule set shared by all B; 1: one set per env */
    int32_t max_episode_steps;  /* L >= 0; 0 = episodes end only when the player is gone */
    int32_t device;             /* HIP device ordinal */
    int32_t engine;             /* av_engine */
    int32_t rule_mode;          /* av_rule_mode */
    void *stream;               /* hipStream_t for all device work; NULL = null stream */
} av_config;

/* Read-only facts about a batch, for callers that use the packed state directly. */
typedef struct {
    int32_t num_envs, height, width, channels;
    int32_t row_bytes;          /* bytes per packed map row: 2 (W <= 16), 4 (W <= 32), 8 */
    int32_t engine;             /* av_engine chosen for av_step / av_step_n */
    size_t state_bytes;         /* size of the packed state behind av_state_ptr */
    size_t blob_bytes;          /* size av_get_state needs */
} av_info;

/* Create a batch of B independent environments on cfg->device (paper Sec. 2.1: a game is a
 * board of C binary tile channels over H x W cells; Sec. 2.3: many environments are stepped
 * in parallel on the accelerator).  Maps start empty; av_load_rules and av_reset must both
 * be called before the first step.  Fails with AV_EINVAL for sizes outside the limits in
 * av_config, when one environment's working set (its C + 1 planes and one match plane per
 * rule, 64-bit rows for W > 32) exceeds 64 KiB of LDS, or when an explicitly requested
 * engine cannot take the configuration (the limits given with av_engine). */
av_status av_create_batch(const av_config *cfg, av_batch_t *out);

/* Load the rules (paper Sec. 2.1: a rule is an n x m input pattern I, an n x m output
 * pattern O, and a reward paid per application, Sec. 2.2.1).  All pointers are host memory
 * and are copied; S = B if per_env_rules else 1; R = num_rules in [0, max_rules].
 *   shape   int32 [S][R][2]: (n rows, m cols), 1 <= n <= min(H, max_pat_h), likewise m
 *   in_pat  int8  [S][R][C+1][max_pat_h][max_pat_w]: 1 must be 1, 0 must be 0, -1 don't care
 *   out_pat int8  same layout: 1 becomes 1, 0 becomes 0, -1 left alone
 *   reward  int32 [S][R]
 * Entries outside a rule's n x m are ignored but must still be in {-1, 0, 1}.  Channel C
 * of a pattern is the force plane.  AV_EINVAL if any set could produce a step reward of
 * magnitude >= 2^24 (sum over rules of |reward| x anchors), which keeps the float reward
 * exact.  Synchronises the stream; replaces any earlier rules for later steps. */
av_status av_load_rules(av_batch_t b, int32_t num_rules, const int32_t *shape,
                        const int8_t *in_pat, const int8_t *out_pat, const int32_t *reward);

/* Site order of rule application control (av_set_rule_control). */
typedef enum {
    AV_SITES_ROW_MAJOR = 0,   /* a capped rule keeps its first matches in row-major order */
    AV_SITES_RANDOM = 1       /* ... the matches with the largest random index value */
} av_site_order;

/* Rule application control (paper Sec. 2.1.1: a rule can be made to apply only once or a
 * fixed number of times, in an ordered or a random order, by taking the maximum over an
 * extra channel of index values; masks let some rules inhibit others).  Applies to the
 * loaded rules only (the four moves are never capped or inhibited).  Per loaded rule, in
 * index order, every step: its matches whose n x m patch overlaps the patch of an applied
 * match of an inhibiting earlier rule are dropped; of the rest at most limit are kept,
 * those with the largest index value; rewards and votes use the kept matches.
 *   limit    host int32 [S][R] or NULL (all 0): 0 = every match applies, K > 0 = at most K
 *   inhibit  host uint8 [S][R][R] or NULL (none): inhibit[s][q][r] != 0 means rule q
 *            inhibits rule r; only q < r is allowed (rule index is priority)
 *   order    av_site_order.  Index value of anchor pos = y * W + x: row-major rank
 *            4095 - pos; random: the high 20 bits of 32-bit word pos % 8 (low half of each
 *            64-bit word first) of Philox4x64-10 (Salmon et al., SC 2011) with counter
 *            (pos / 8, n, env, 0) and key (seed, 0), above that rank, where n is the batch
 *            step number (steps since av_reset, all environments counted together)
 *   seed     key of the random index channel
 * Engines: on a lane16 batch the control is compiled into the lane16 program (a new
 * program per call); the wave engine runs it when its scratch (about 1.3 KiB, plus 4 bytes
 * per cell for the random channel) still fits its 64 KiB of LDS.  A batch created with
 * AV_ENGINE_AUTO whose engine is group or rows switches to the wave engine on those terms,
 * and otherwise to the generic engine, while some limit or inhibition is set; explicit group
 * and rows batches refuse the control, and so does an explicit wave batch whose scratch does
 * not fit (AV_EINVAL).
 * AV_ESTATE before av_load_rules (which clears the control); AV_EINVAL for a negative
 * limit, an inhibition with q >= r or an unknown order.  Synchronises the stream. */
av_status av_set_rule_control(av_batch_t b, const int32_t *limit, const uint8_t *inhibit,
                              int32_t order, uint64_t seed);

/* Set every environment's initial map and current map to init_maps (device, uint8
 * [B][C][H][W], nonzero = tile present), its step counter and the batch step number to 0
 * (paper Sec. 2.2.1: an environment is its initial layout and its rules; Sec. 2.3: an episode
 * that ends restarts from the initial layout).  Environments that end an episode return to
 * these maps.  Rules (av_load_rules) and maps may be given in either order.  May
 * synchronise. */
av_status av_reset(av_batch_t b, const uint8_t *init_maps);

/* One step of all B environments (paper Sec. 2.1: the action places force tiles next to the
 * player, every rule is matched by a thresholded convolution with its input pattern and its
 * output written by a transposed convolution; Sec. 2.1.1: the rules apply in parallel, or
 * per av_config.rule_mode; Sec. 2.2.1: rules pay rewards, and a step that leaves no player
 * ends the episode).  actions: device uint8 [B] (0 none, 1 up, 2 right, 3 down, 4 left,
 * other values as 0); rewards: device float [B] (exact small integers); done: device uint8
 * [B] (0/1).  AV_ESTATE before av_load_rules and av_reset.  Asynchronous; a launch made on a
 * capturing stream (av_set_stream) can be replayed from a HIP graph: the batch step number
 * is kept on the device and advances on every replay. */
av_status av_step(av_batch_t b, const uint8_t *actions, float *rewards, uint8_t *done);

/* k consecutive steps in one launch, identical in result to k calls of av_step (the same
 * step, paper Sec. 2.1, Sec. 2.1.1, Sec. 2.2.1, repeated as the learning loop of Sec. 2.3
 * steps its environments).  actions uint8 [k][B], rewards float [k][B], done uint8 [k][B],
 * all device; k >= 1.  Maps stay on chip between the k steps.  AV_ESTATE before
 * av_load_rules and av_reset.  Asynchronous (capturable as av_step). */
av_status av_step_n(av_batch_t b, int32_t k, const uint8_t *actions, float *rewards,
                    uint8_t *done);

/* k steps (as av_step_n) followed by the observation of the resulting maps (as av_observe,
 * paper Sec. 2.2.2), for agents that act on every step's observation.  On the lane16 engine
 * with w <= 12 the window is written by the step kernel itself from the maps it holds in
 * registers (one launch, no re-read of the maps); otherwise the observation kernel follows
 * the step on the same stream.  obs: device uint8 [B][C][w][w], w in [1, 255].
 * Asynchronous. */
av_status av_step_observe(av_batch_t b, int32_t k, const uint8_t *actions, float *rewards,
                          uint8_t *done, int32_t w, uint8_t *obs);

/* Current maps as device uint8 [B][C][H][W] (0/1) written to dst.  Asynchronous. */
av_status av_get_maps(av_batch_t b, uint8_t *dst);

/* The player-centred observation of the current maps (paper Sec. 2.2.2: a local patch of
 * tiles centred on the player's position; Table 1 uses windows of 5, 10, 20 and 31 cells).
 * dst: device uint8 [B][C][w][w], w in [1, 255].  Window cell (wy, wx) shows map cell
 * (py - w/2 + wy, px - w/2 + wx), where (py, px) is the environment's first player cell in
 * row-major order and w/2 is rounded down; cells off the map, and the whole window of an
 * environment without a player, are 0.  Asynchronous. */
av_status av_observe(av_batch_t b, int32_t w, uint8_t *dst);

/* The loaded rules as binary features (paper Sec. 2.2.2: the agent also observes a binary
 * representation of its environment's rules).  dst: device uint8
 * [S][R][2][2][C+1][max_pat_h][max_pat_w] with S = B if per_env_rules else 1: index 2 is
 * 0 input / 1 output pattern, index 3 is 0 "entry specified" / 1 "entry value" (0 when not
 * specified).  AV_ESTATE before av_load_rules.  May synchronise. */
av_status av_rule_features(av_batch_t b, uint8_t *dst);

/* Mutation operators (paper Sec. 2.2.1 and the Fig. 2b caption: environments are mutated by
 * flipping bits of the initial multi-hot map, by changing entries of the rules' input and
 * output patterns, and by changing the rules' rewards), batched over a population of
 * individuals.  They work on caller-owned device arrays in the layouts av_reset and
 * av_load_rules take (so a generation is mutated on the GPU and then loaded), need no batch,
 * and run on `stream` of `device`; asynchronous.  Destinations may equal their sources.
 *
 * Randomness: a 32-bit word w of stream t for individual k is half (w % 2, low half first)
 * of 64-bit output word (w % 8) / 2 of Philox4x64-10 (Salmon et al., SC 2011) at counter
 * (w / 8, generation, k, t) with key (seed, 0).  An event with threshold p (a *_p32 field)
 * happens iff its word is < p, i.e. with probability p / 2^32. */
typedef struct {
    uint64_t seed;              /* key of every stream */
    uint64_t generation;        /* counter word: a fresh draw per generation */
    uint32_t map_flip_p32;      /* per map bit (stream 1) */
    uint32_t map_channels;      /* bit c set: map channel c may flip */
    uint32_t entry_p32;         /* per pattern entry inside its rule's n x m (stream 2) */
    uint32_t entry_channels;    /* bit c set: pattern channel c (C = force) may change */
    uint32_t reward_p32;        /* per rule reward (stream 3) */
    int32_t reward_lo, reward_hi; /* a redrawn reward is uniform-by-modulo in [lo, hi] */
} av_mutation;

/* Map mutation: src, dst device uint8 [n][C][H][W] (nonzero = tile; dst gets 0/1).  Bit
 * e = (c * H + y) * W + x of individual k flips iff bit c of map_channels is set and word e
 * of stream 1 is below map_flip_p32.  n >= 0; C in [1, 31]; H, W in [1, 64].  AV_EINVAL for a
 * NULL pointer (with n > 0), sizes out of range or m == NULL; AV_EDEVICE on a launch
 * failure. */
av_status av_mutate_maps(const uint8_t *src, uint8_t *dst, int32_t n, int32_t channels,
                         int32_t height, int32_t width, const av_mutation *m, int32_t device,
                         void *stream);

/* Rule mutation in the av_load_rules layout, all device arrays: shape int32 [S][R][2],
 * in/out patterns int8 [S][R][C+1][max_pat_h][max_pat_w], rewards int32 [S][R]; individual
 * = set s.  Entry e = (((r * 2 + io) * (C + 1) + c) * max_pat_h + i) * max_pat_w + j (io 0 =
 * input, 1 = output) with i < n, j < m of its rule and bit c of entry_channels set changes
 * iff word 2e of stream 2 is below entry_p32; it then takes the lower (word 2e + 1 even) or
 * higher (odd) of the two values of {-1, 0, 1} other than its own (a value outside that set
 * counts as 1).  Reward r is redrawn iff word 2r of stream 3 is below reward_p32, to
 * reward_lo + (word 2r + 1) mod (reward_hi - reward_lo + 1).  Mutated rewards are not
 * checked against the 2^24 bound here; av_load_rules checks them.  AV_EINVAL for NULL
 * pointers (with S * R > 0), sizes out of range (S >= 0; R in [0, 252]; C in [1, 31]; pattern
 * extents in [1, 16]), reward_lo > reward_hi or m == NULL. */
av_status av_mutate_rules(int32_t num_sets, int32_t num_rules, int32_t channels,
                          int32_t max_pat_h, int32_t max_pat_w, const int32_t *shape,
                          const int8_t *in_src, const int8_t *out_src, const int32_t *reward_src,
                          int8_t *in_dst, int8_t *out_dst, int32_t *reward_dst,
                          const av_mutation *m, int32_t device, void *stream);

/* ---------------------------------------------------------------------------------------
 * Batched search (paper Sec. 2.2.1: an environment is scored by searching the player's
 * action sequences; a node is a game state — the map, which holds the player's position,
 * and the reward accumulated so far — an edge is an action; a state equal to one seen
 * before keeps the node with the higher reward, then the shallower one).
 *
 * Two orders.  Level order (best_first_k = 0; breadth-first, which the paper also names):
 * one av_search_expand steps every (frontier node, action) pair of the level as one batch
 * with the step engines above.  Batched best-first (best_first_k = k >= 1; the paper's
 * fitness search prioritises higher reward): open nodes are ordered by higher reward, then
 * smaller depth, then smaller node id (the root is node 0, kept children get the next ids in
 * child order); one av_search_expand pops the first k open nodes, drops those whose state
 * has since been reached with a better (reward, -depth), and expands the rest, in id order,
 * exactly like one level below; the kept children are opened.  k = 1 is plain best-first.
 * Level d (or one best-first iteration):
 *   - children: frontier nodes in order, for each the actions in order (0..4, or 1..4 with
 *     num_actions = 4), cut to max_children; child i of a level is visit number
 *     visited + 1 + i (the root is visit 0);
 *   - a child is its parent's map stepped once with its action, its step counter starting
 *     at the parent's depth (so a child of depth max_episode_steps ends its episode); its
 *     reward is the parent's plus the step's; the best node is the one with the highest
 *     reward, earliest visit first (the root, reward 0, counts);
 *   - children whose episode ended are terminal: counted, never expanded;
 *   - the others are deduplicated by state: two children, or a child and an earlier node,
 *     hold the same state iff their maps are equal cell for cell.  A 64-bit hash of the
 *     packed map (SplitMix64's finalizer chained over each channel's rows read as 64-bit
 *     words) only chooses where the state is looked up in the table; maps with equal hashes
 *     are compared and kept apart when they differ.  A child survives iff it has the best
 *     (reward, -depth) of its state in this level, lowest index among equals, and its state
 *     is new or it beats the (reward, -depth) stored for the state; survivors in index
 *     order, cut to max_frontier, are the next frontier.
 * ------------------------------------------------------------------------------------- */
typedef struct av_search_s *av_search_t;

typedef struct {
    int32_t height, width, channels;   /* map shape; limits as av_config */
    int32_t max_rules, max_pat_h, max_pat_w;
    int32_t max_episode_steps;         /* L >= 0; 0 = episodes end only without a player */
    int32_t num_actions;               /* 5 (actions 0..4) or 4 (actions 1..4) */
    int32_t max_frontier;              /* level order: most nodes kept per level, [1, 2^24] */
    int32_t table_log2;                /* hash table of 2^table_log2 slots, in [4, 31] */
    int32_t device, engine, rule_mode; /* as av_config; engine AUTO picks as for a batch */
    int32_t best_first_k;              /* 0: level order; k in [1, 512]: batched best-first */
    int32_t max_nodes;                 /* best-first: node pool capacity, in [1, 2^26] */
    int32_t hash_bits;                 /* 0: the full 64-bit map hash; h in [1, 63]: only its
                                          low h bits (more maps share a hash; results do not
                                          change, since states are compared exactly) */
    void *stream;                      /* hipStream_t; NULL = null stream */
} av_search_config;

typedef struct {
    int64_t level;          /* levels expanded since av_search_begin */
    int64_t parents;        /* frontier nodes this call started from */
    int64_t children;       /* states visited (stepped) by this call */
    int64_t terminal;       /* of them, episode ends */
    int64_t survivors;      /* new or improved states, before the max_frontier cut */
    int64_t frontier;       /* nodes in the frontier now (best-first: open nodes) */
    int64_t visited;        /* states visited since av_search_begin */
    int64_t best_visit;     /* visit number of the best node (0 = the root) */
    int32_t best_reward;    /* its accumulated reward */
    int32_t reserved;
} av_search_info;

/* Create a search: a children batch of num_actions x max_frontier environments, frontier
 * buffers and the state table (28 bytes per slot plus the slot's packed map, C x H x
 * row_bytes bytes, where row_bytes is 2, 4 or 8 for W up to 16, 32 or 64) on cfg->device.
 * AV_EINVAL for sizes out of range, AV_ENOMEM if the device allocations fail. */
av_status av_search_create(const av_search_config *cfg, av_search_t *out);

/* The rule set searched (one set, host arrays, layouts and checks as av_load_rules with
 * S = 1).  Synchronises. */
av_status av_search_load_rules(av_search_t s, int32_t num_rules, const int32_t *shape,
                               const int8_t *in_pat, const int8_t *out_pat,
                               const int32_t *reward);

/* Start from root (device uint8 [C][H][W], nonzero = tile): frontier = {root} at depth 0
 * and reward 0, table = {root}, no visits.  AV_ESTATE before av_search_load_rules. */
av_status av_search_begin(av_search_t s, const uint8_t *root);

/* Expand one level (above) with at most max_children >= 0 children; fills *info (host).
 * An empty frontier or max_children = 0 expands nothing and keeps the frontier.  A search
 * visits at most 2^32 - 2 states (AV_EINVAL beyond).
 * Synchronises once, after the children are posted (the next level's size is needed on the
 * host); the level's last copies may still run on the search's stream when it returns (later
 * calls on the search are ordered after them).  AV_ENOMEM when an insertion
 * finds 4096 consecutive slots taken by other keys (the table is too full) or, best-first,
 * when the node pool is full: the search must then be restarted with av_search_begin. */
av_status av_search_expand(av_search_t s, int64_t max_children, av_search_info *info);

/* The current frontier (level order) or the open list in priority order (best-first):
 * maps device uint8 [N][C][H][W], reward and depth device int32 [N], N = info.frontier; any
 * pointer may be NULL to skip it.  Asynchronous. */
av_status av_search_frontier(av_search_t s, uint8_t *maps, int32_t *reward, int32_t *depth);

/* Free the search; NULL is a no-op.  Synchronises. */
av_status av_search_destroy(av_search_t s);

/* For callers that cannot allocate device memory (harnesses that forbid hipMalloc, tight
 * serving loops): k steps of B caller-owned environments, with the results of av_step_n on a
 * batch made with *cfg, loaded with these rules and holding this state, on the wave engine
 * (AV_ENGINE_WAVE, or AV_ENGINE_AUTO when its LDS working set fits) or the generic engine
 * (AV_ENGINE_GENERIC, or AUTO otherwise).  Nothing is allocated: the compiled rule program and
 * the launch units' scratch (8 bytes per environment) live in a static device array of the
 * library of AV_STATIC_SCRATCH_BYTES per device, held until the process ends.
 *   cfg       as av_create_batch (device, stream, sizes, per_env_rules, L, rule_mode); engine
 *             AUTO, WAVE or GENERIC; no rule application control
 *   rules     host arrays in the av_load_rules layout and with its checks
 *   state     device, packed current maps [C][B][H] rows of row_bytes (2, 4 or 8 bytes for W
 *             up to 16, 32, 64; bit x = column x), the layout of av_state_ptr; read and written
 *   init      device, packed initial maps, same layout; episodes that end return to them
 *   counters  device int32 [B], each environment's step counter; read and written
 *   actions, rewards, done   as av_step_n ([k][B], device)
 * AV_EINVAL (before any device work) for sizes out of range, NULL pointers, k < 1, bad rules,
 * or a scratch image (8 x (B + 8) bytes plus the compiled program) above
 * AV_STATIC_SCRATCH_BYTES.  Every call on one device shares that device's array and leaves
 * the last program in it: calls that overlap on one device (other streams, other threads)
 * race.  The program is copied from pageable host memory on the stream, which waits for the
 * stream's earlier work; the call cannot be captured into a graph. */
#define AV_STATIC_SCRATCH_BYTES (4u << 20)
av_status av_step_n_static(const av_config *cfg, int32_t num_rules, const int32_t *shape,
                           const int8_t *in_pat, const int8_t *out_pat, const int32_t *reward,
                           void *state, const void *init, int32_t *counters, int32_t k,
                           const uint8_t *actions, float *rewards, uint8_t *done);

/* Device pointer to the packed current maps, owned by the batch and valid until the
 * next av_reset / av_set_state / av_destroy_batch.  Layout: rows of row_bytes bytes,
 * index [c][env][y] (channel-major over the whole batch); cell (env, c, y, x) is bit x
 * (least significant first) of that row.  NULL on error. */
const void *av_state_ptr(av_batch_t b);

av_status av_get_info(av_batch_t b, av_info *info);

/* Checkpoint and resume.  av_get_state copies the packed current maps, initial maps, step
 * counters and the batch step number into host_blob; *bytes holds its capacity on entry and the size written
 * on return (call with host_blob = NULL to query).  av_set_state restores them; stepping
 * on from a restored blob is bit-identical to stepping on from where it was taken.  The
 * blob records B, H, W, C and is refused (AV_EINVAL) by a batch of another shape.
 * Both synchronise. */
av_status av_get_state(av_batch_t b, void *host_blob, size_t *bytes);
av_status av_set_state(av_batch_t b, const void *host_blob, size_t bytes);

/* Change the stream later calls use (hipStream_t; NULL = null stream). */
av_status av_set_stream(av_batch_t b, void *stream);

/* Free all device and host state of the batch; synchronises its stream.  NULL is a no-op. */
av_status av_destroy_batch(av_batch_t b);

/* Message for the last failing call on this thread; "" if none.  Never NULL. */
const char *av_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* AUTOVERSE_H */
