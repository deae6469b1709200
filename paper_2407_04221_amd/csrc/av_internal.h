// Internal declarations of libautoverse: the compiled rule program, the batch object and
// the kernel launchers.  Not part of the public ABI (include/autoverse.h).
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/autoverse.h"

namespace av {

// Tile roles (paper Sec. 2.2.1, base maze game).
constexpr int kChEmpty = 0, kChWall = 1, kChPlayer = 2, kChGoal = 3;
constexpr int kMoveRules = 4;     // built-in moves, rule indices 0..3 of every set
constexpr int kMaxRules = 252;    // loaded rules; with the moves a rule index fits a byte
constexpr int kMaxDim = 64;       // largest H and W
constexpr int kMaxPat = 16;       // largest pattern rows / cols
constexpr int kLdsBudget = 64 * 1024;
constexpr int kFusedObserveMax = 12;   // largest window the lane16 step kernel writes itself

// ---------------------------------------------------------------------------------
// Compiled rules, generic form.  Built on the host from the tri-valued patterns; one
// "set" per environment or one shared set.  Every set starts with the four moves.
//
// Match entry (one specified input entry): bits 0-7 channel, 8-15 row i, 16-23 col j,
// bit 24 wanted value.  Vote entry (one nonzero K_O entry), grouped by channel:
// bits 0-7 rule, 8-15 row i, 16-23 col j, bit 24 set when the vote is +1.  Rule-major
// vote entry (the same votes grouped by rule; the force plane's are left out in parallel
// mode, where the plane is dropped before anything reads it again): bits 0-7 channel,
// 8-15 row i, 16-23 col j, bit 24 set for +1.
// ---------------------------------------------------------------------------------
struct RuleHdr {
    int32_t n, m;         // pattern rows, cols
    int32_t reward;
    int32_t match_off;    // into the set's match entries
    int32_t match_cnt;
    int32_t vote_off;     // into the set's rule-major vote entries
    int32_t vote_cnt;
    int32_t pad;          // bit c: some rule-major vote of the rule is on channel c (c < 32)
};

struct VoteList {
    int32_t off, cnt;     // into the set's vote entries
};

struct GenericProgram {
    int32_t rules_per_set = 0;        // R + 4
    int32_t sets = 0;                 // S
    int32_t match_stride = 0;         // match entries per set (max over sets)
    int32_t vote_stride = 0;          // vote entries per set (max over sets)
    int32_t any_reward = 0;
    std::vector<RuleHdr> hdr;         // [S][R+4]
    std::vector<VoteList> votes;      // [S][C+1]
    std::vector<uint32_t> match;      // [S][match_stride]
    std::vector<uint32_t> vote;       // [S][vote_stride]
    int32_t rvote_stride = 0;         // rule-major vote entries per set (max over sets)
    std::vector<uint32_t> rvote;      // [S][rvote_stride]
};

inline uint32_t pack_match(int c, int i, int j, int want) {
    return uint32_t(c) | (uint32_t(i) << 8) | (uint32_t(j) << 16) | (uint32_t(want) << 24);
}
inline uint32_t pack_vote(int r, int i, int j, bool plus) {
    return uint32_t(r) | (uint32_t(i) << 8) | (uint32_t(j) << 16) | (uint32_t(plus) << 24);
}

// One rule in tri-valued form over C + 1 channels, n x m (1 must be 1, 0 must be 0,
// -1 don't care).
struct HostRule {
    int n = 1, m = 1, reward = 0;
    std::vector<int8_t> in, out;   // [C+1][n][m]
    int8_t at(const std::vector<int8_t> &p, int c, int i, int j) const {
        return p[(size_t(c) * n + i) * m + j];
    }
};

// Host-side rule handling (av_api.cpp): the checked rule sets of av_load_rules' arguments
// (each starting with the four moves; failures set the thread's last error), and their
// compiled generic program (rule-major votes include the force plane's when force_votes).
av_status parse_rule_sets(const av_config &c, int32_t R, const int32_t *shape,
                          const int8_t *in_pat, const int8_t *out_pat, const int32_t *reward,
                          std::vector<std::vector<HostRule>> &sets);
void compile_generic(const std::vector<std::vector<HostRule>> &sets, int C, bool force_votes,
                     GenericProgram &p);

// Device-side copy of a generic program.
struct DeviceProgram {
    RuleHdr *hdr = nullptr;
    VoteList *votes = nullptr;
    uint32_t *match = nullptr;
    uint32_t *vote = nullptr;
    uint32_t *rvote = nullptr;
    int32_t rules_per_set = 0, match_stride = 0, vote_stride = 0, rvote_stride = 0;
    int32_t any_reward = 0;           // some rule of some set pays a nonzero reward
    // group engine only (k_group.hip): per set, the probe table and the channel vote lists'
    // rule ranges, gtab_stride words each, and the input entries merged per plane row,
    // gmatch_stride words each
    uint32_t *gtab = nullptr;
    int32_t gtab_stride = 0;
    uint32_t *gmatch = nullptr;
    int32_t gmatch_stride = 0;
};

// Rule application control (paper Sec. 2.1.1): per loaded rule a cap on the matches applied
// per step, chosen by the largest index-channel value, and rules that inhibit later ones.
// Arrays are indexed by the set's internal rule index (moves 0..3 carry no control).
struct CtlArgs {
    const int32_t *limit = nullptr;     // [S][R+4]; 0 = every match applies
    const uint32_t *inhibit = nullptr;  // [S][R+4][words]; bit q of rule r: q inhibits r
    int32_t words = 0;                  // inhibitor mask words per rule
    int32_t active = 0;                 // some limit or inhibition is set
    int32_t random = 0;                 // index channel: 0 row-major rank, 1 random
    uint64_t seed = 0;                  // key of the random index channel
};

// Everything a step kernel needs, passed by value.
struct StepArgs {
    int32_t B, H, W, C, L;
    int32_t per_env;
    int32_t sequential;              // rules applied one after another (else in parallel)
    int32_t k;                       // steps in this launch
    int32_t row_bytes;
    int32_t max_pat_h = 1;           // largest pattern rows a loaded rule may have
    int32_t max_pat_w = 1;           // largest pattern columns
    // group engine: workgroup i steps environment order[i] (null: environment i) and, when cost
    // is set, records the cycles its wave took in cost[environment] / 256
    const int32_t *order = nullptr;
    uint32_t *cost = nullptr;
    void *state;                     // [C][B][H] rows
    const void *init;                // [C][B][H] rows
    int32_t *t;                      // [B] step counters
    // Batch step numbers (steps since av_reset, the random index channel's counter word),
    // one copy per launch unit: per wave on lane16, per workgroup on the other engines.
    // Every unit reads its copy at the start of a launch and stores it advanced by k at the
    // end, so the number lives on the device and captured launches replay correctly; all
    // copies a unit index reaches hold the same value (av_api re-broadcasts copy 0 whenever
    // the engine or its launch shape changes).  B + 8 entries.
    uint64_t *nctr;
    const uint8_t *actions;          // [k][B]
    float *rewards;                  // [k][B]
    uint8_t *done;                   // [k][B]
    DeviceProgram prog;
    CtlArgs ctl;
    uint8_t *obs = nullptr;          // lane16 only: observation of the final maps, [B][C][w][w]
    int32_t obs_w = 0;               // window size, <= 64
    // lane16 only, search expansion: environment e starts from row block e / gA of gsrc
    // ([C][gnf][H]) with counter gdepth[e / gA] and no initial maps
    const void *gsrc = nullptr;
    int32_t gnf = 0, gA = 1;
    const int32_t *gdepth = nullptr;
};

// Launchers (k_generic.hip).  All return hipSuccess or the launch error.
hipError_t launch_pack(const uint8_t *src, void *dst, void *dst2, int B, int C, int H, int W,
                       int row_bytes, hipStream_t s);
hipError_t launch_unpack(const void *src, uint8_t *dst, int B, int C, int H, int W,
                         int row_bytes, hipStream_t s);
// Step counters and batch step numbers without hipMemsetAsync (a fill kernel is safe under
// stream capture): t[0..B) = 0 when t is given; nctr[0..n) = value, or = nctr[0] when
// broadcast is set.
hipError_t launch_fill_counters(int32_t *t, int B, uint64_t *nctr, int n, int broadcast,
                                uint64_t value, hipStream_t s);
hipError_t launch_generic_step(const StepArgs &a, int envs_per_block, hipStream_t s);
size_t generic_env_lds_bytes(int H, int W, int C, int rules_per_set, bool control = false,
                             bool random = false);

// Mutation operators (k_mutate.hip); MutateArgs mirrors av_mutation.
struct MutateArgs {
    uint64_t seed, generation;
    uint32_t map_flip_p32, map_channels;
    uint32_t entry_p32, entry_channels;
    uint32_t reward_p32;
    int32_t reward_lo, reward_hi;
};
hipError_t launch_mutate_maps(const uint8_t *src, uint8_t *dst, int n, int C, int H, int W,
                              const MutateArgs &m, hipStream_t s);
hipError_t launch_mutate_rules(int S, int R, int C, int mh, int mw, const int32_t *shape,
                               const int8_t *in_src, const int8_t *out_src,
                               const int32_t *reward_src, int8_t *in_dst, int8_t *out_dst,
                               int32_t *reward_dst, const MutateArgs &m, hipStream_t s);

// Batched search (k_search.hip, av_search.cpp).  One level's device arrays and sizes.
struct SearchArgs {
    int32_t n = 0, A = 5, C = 0, H = 0, cap = 0;   // children, actions, channels, rows, frontier cap
    uint64_t visited = 0;                          // visits before this level
    uint32_t cur_epoch = 0;                        // this level's stamp (levels count from 1)
    const int32_t *front_reward = nullptr, *front_depth = nullptr;   // [nf]
    const float *rew = nullptr;                    // [n] step rewards of the children
    const uint8_t *done = nullptr;                 // [n]
    int32_t *kid_reward = nullptr, *kid_depth = nullptr;             // [n]
    uint64_t *kid_val = nullptr;                   // [n] packed (reward, -depth)
    int64_t *slot = nullptr;                       // [n] table slot, -1 if none
    uint64_t *keys = nullptr, *vals = nullptr, *claim = nullptr;     // [slots]
    uint32_t *epoch = nullptr;                     // [slots]
    void *store = nullptr;                         // [slots][C][H] rows: each slot's map
    uint64_t mask = 0;                             // slots - 1
    uint64_t hash_mask = ~0ull;                    // bits of the map hash that are used
    uint64_t *best = nullptr;                      // packed (reward, -visit)
    uint32_t *counts = nullptr;                    // terminal, overflow, survivors
    int32_t *block_count = nullptr;                // [ceil(n / 256)]
    int32_t *src_of = nullptr;                     // [cap] child of each next-frontier node
    int32_t *next_reward = nullptr, *next_depth = nullptr;           // [cap]
    void *next = nullptr;                          // next frontier rows [C][next_n][H]
    int32_t next_n = 0, next_off = 0;              // its block count and first block written
    int64_t *root_slot = nullptr;                  // root_kernel: the root's table slot
};
// phase 0 gather, 1 post/claim/flag/scan/place, 2 copy rows (nn nodes), 3 root insert.
hipError_t launch_search_phase(const SearchArgs &a, int row_bytes, const void *front, int nf,
                               void *kids, int32_t *kid_t, hipStream_t s, int phase, int nn);

// Batched best-first pieces (k_search.hip).
hipError_t launch_copy_rows(int row_bytes, const void *src, int nsrc, const int32_t *src_of,
                            void *dst, int ndst, int off, int n, int C, int H, hipStream_t s);
hipError_t launch_bf_pop(const uint32_t *open_ids, int kp, const int64_t *pool_slot,
                         const uint64_t *pool_val, const uint64_t *vals, int32_t *parents,
                         uint32_t *n_par, uint32_t *counts, hipStream_t s);
hipError_t launch_bf_gather_meta(const int32_t *parents, int np, const int32_t *pool_reward,
                                 const int32_t *pool_depth, int32_t *front_reward,
                                 int32_t *front_depth, hipStream_t s);
hipError_t launch_bf_append(const int32_t *src_of, int nn, int pool_n, const uint64_t *kid_val,
                            const int64_t *slot, uint64_t *pool_val, int64_t *pool_slot,
                            uint64_t *new_keys, uint32_t *new_ids, hipStream_t s);
hipError_t launch_bf_merge(const uint64_t *ok, const uint32_t *oi, int m, const uint64_t *nk,
                           const uint32_t *ni, int nn, uint64_t *outk, uint32_t *outi,
                           hipStream_t s);
hipError_t launch_bf_open(int row_bytes, const void *pool, int pcap, const uint32_t *ids, int n,
                          int C, int H, int W, uint8_t *maps, const int32_t *pool_reward,
                          const int32_t *pool_depth, int32_t *reward, int32_t *depth,
                          hipStream_t s);

// Internal access to a batch for the search (av_api.cpp).
void *batch_state(av_batch_t b);
int32_t *batch_counters(av_batch_t b);
int batch_row_bytes(av_batch_t b);
// One step of the first n environments of b, whose state rows are laid out [C][n][H].
// With gsrc (lane16 batches only), environment e's rows are read from block e / gA of gsrc
// ([C][gnf][H]) and its counter from gdepth[e / gA] instead.
av_status step_prefix(av_batch_t b, int n, const uint8_t *actions, float *rewards,
                      uint8_t *done, const void *gsrc = nullptr, int gnf = 0, int gA = 1,
                      const int32_t *gdepth = nullptr);
int batch_engine(av_batch_t b);
av_status set_error(av_status st, const char *msg);

// Player-centred observation window (k_observe.hip).
hipError_t launch_observe(const void *state, int B, int C, int H, int W, int row_bytes, int w,
                          uint8_t *dst, hipStream_t s);

// The rows engine (k_rows.hip): one environment per wave, planes in registers, and its
// program: per set, rule headers, probe and row-ordered match entries, row-ordered votes.
struct RowsProgram {
    int32_t rules = 0, sets = 0, set_words = 0;
    std::vector<uint32_t> words;      // [S][set_words]
};
void compile_rows(const GenericProgram &g, int C, RowsProgram &out);
size_t rows_lds_bytes(int H, int W, int C, int rules_per_set);
bool rows_eligible(int H, int W, int C, int rules_per_set);
hipError_t launch_rows_step(const StepArgs &a, const uint32_t *words, int set_words, int rules,
                            hipStream_t s);

// The group engine (k_group.hip): one environment per wave, its rules dealt to 2 or 4 groups
// of lanes; parallel rule order, no rule application control.
bool group_eligible(int H, int W, int C, int rules_per_set, int max_pat_h, int max_pat_w);
// The group engine's per-set tables (probe rows of the loaded rules, rule ranges of the
// channel vote lists) for maps of H x W with patterns of up to max_pat_h rows, laid out as
// the kernel keeps them in LDS, and its input entries merged per plane row (gm, gm_stride
// words per set).
void compile_group_tables(const GenericProgram &p, int H, int W, int C, int max_pat_h,
                          std::vector<uint32_t> &tab, int &stride, std::vector<uint32_t> &gm,
                          int &gm_stride);
hipError_t launch_group_step(const StepArgs &a, hipStream_t s);

// Wave slots of the current device (8 waves per SIMD, 4 SIMDs per CU; 0 if it cannot be
// asked): the most waves resident at once.
long long device_wave_slots();

// The wave engine (k_wave.hip): one environment per workgroup.
size_t wave_lds_bytes(int H, int W, int C, int rules_per_set, bool control = false,
                      bool random = false);
hipError_t launch_wave_step(const StepArgs &a, hipStream_t s);

}  // namespace av
