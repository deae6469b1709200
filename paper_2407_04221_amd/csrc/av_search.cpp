// Batched search (include/autoverse.h, av_search_*): host side.  Owns a children batch
// (stepped with the batch engines), two frontier buffers, the hash table and the per-level
// scratch arrays; each level runs gather -> step -> post/claim/flag/scan/place -> copy on the
// search's stream with one synchronisation to learn the next frontier's size.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <new>
#include <vector>

#include "av_internal.h"

using namespace av;

struct av_search_s {
    av_search_config cfg{};
    hipStream_t stream = nullptr;
    av_batch_t kids = nullptr;       // num_actions x max_frontier environments
    int row_bytes = 0;
    int A = 5;
    int64_t cap = 0;                 // max_frontier
    uint64_t slots = 0;
    void *front[2] = {nullptr, nullptr};
    int32_t *reward[2] = {nullptr, nullptr}, *depth[2] = {nullptr, nullptr};
    int cur = 0;                     // which frontier buffer is current
    int64_t n_front = 0;
    uint8_t *actions = nullptr;      // [A * cap]: child i takes action i % A (+1 for A = 4)
    float *rew = nullptr;
    uint8_t *done = nullptr;
    int32_t *kid_reward = nullptr, *kid_depth = nullptr, *block_count = nullptr, *src_of = nullptr;
    uint64_t *kid_val = nullptr;
    int64_t *slot = nullptr;
    uint64_t *keys = nullptr, *vals = nullptr, *claim = nullptr, *best = nullptr;
    uint32_t *epoch = nullptr, *counts = nullptr;
    void *store = nullptr;           // [slots][C][H] rows: the map of each slot's state
    bool have_rules = false, begun = false;
    int64_t level = 0, visited = 0;
    // batched best-first (K > 0): node pool, open list (value, id) sorted, popped parents
    int K = 0;
    int64_t pcap = 0, pool_n = 0, open_n = 0;
    void *pool = nullptr;
    int32_t *pool_reward = nullptr, *pool_depth = nullptr, *parents = nullptr;
    uint64_t *pool_val = nullptr, *new_keys = nullptr;
    int64_t *pool_slot = nullptr;
    uint64_t *okeys[2] = {nullptr, nullptr};
    uint32_t *oids[2] = {nullptr, nullptr}, *new_ids = nullptr, *n_par = nullptr;
    int ocur = 0;
};

namespace {

#define SEARCH_HIP(call)                                                                 \
    do {                                                                                 \
        hipError_t e_ = (call);                                                          \
        if (e_ != hipSuccess) {                                                          \
            char m_[256];                                                                \
            std::snprintf(m_, sizeof m_, "%s failed: %s", #call, hipGetErrorString(e_)); \
            return set_error(e_ == hipErrorOutOfMemory ? AV_ENOMEM : AV_EDEVICE, m_);    \
        }                                                                                \
    } while (0)

template <typename T>
hipError_t alloc(T **p, size_t count) {
    return hipMalloc(reinterpret_cast<void **>(p), std::max<size_t>(count, 1) * sizeof(T));
}

void release(av_search_t s) {
    void *ptrs[] = {s->front[0], s->front[1], s->reward[0], s->reward[1], s->depth[0], s->depth[1],
                    s->actions, s->rew, s->done, s->kid_reward, s->kid_depth, s->block_count,
                    s->src_of, s->kid_val, s->slot, s->keys, s->vals, s->claim, s->best, s->epoch,
                    s->counts, s->store, s->pool, s->pool_reward, s->pool_depth, s->parents,
                    s->pool_val,
                    s->new_keys, s->pool_slot, s->okeys[0], s->okeys[1], s->oids[0], s->oids[1],
                    s->new_ids, s->n_par};
    for (void *p : ptrs)
        if (p) (void)hipFree(p);
    if (s->kids) av_destroy_batch(s->kids);
}

SearchArgs level_args(av_search_t s, int n) {
    SearchArgs a;
    a.n = n; a.A = s->A; a.C = s->cfg.channels; a.H = s->cfg.height; a.cap = int(s->cap);
    a.visited = uint64_t(s->visited);
    a.cur_epoch = uint32_t(s->level + 1);
    a.front_reward = s->reward[s->cur]; a.front_depth = s->depth[s->cur];
    a.rew = s->rew; a.done = s->done;
    a.kid_reward = s->kid_reward; a.kid_depth = s->kid_depth; a.kid_val = s->kid_val;
    a.slot = s->slot;
    a.keys = s->keys; a.vals = s->vals; a.claim = s->claim; a.epoch = s->epoch;
    a.store = s->store;
    a.mask = s->slots - 1;
    a.hash_mask = s->cfg.hash_bits == 0 ? ~0ull : (1ull << s->cfg.hash_bits) - 1;
    a.best = s->best; a.counts = s->counts;
    a.block_count = s->block_count; a.src_of = s->src_of;
    a.next_reward = s->reward[1 - s->cur]; a.next_depth = s->depth[1 - s->cur];
    a.next = s->front[1 - s->cur];
    return a;
}

// best node word: (reward with its sign bit flipped) << 32 | ~visit
av_status decode_best(uint64_t best, av_search_info *info) {
    info->best_reward = int32_t(uint32_t(best >> 32) ^ 0x80000000u);
    info->best_visit = int64_t(0xFFFFFFFFull - (best & 0xFFFFFFFFull));
    return AV_OK;
}

av_status read_best(av_search_t s, av_search_info *info) {
    uint64_t best = 0;
    SEARCH_HIP(hipMemcpyAsync(&best, s->best, sizeof best, hipMemcpyDeviceToHost, s->stream));
    SEARCH_HIP(hipStreamSynchronize(s->stream));
    return decode_best(best, info);
}

}  // namespace

extern "C" {

av_status av_search_create(const av_search_config *cfg, av_search_t *out) {
    if (!out) return set_error(AV_EINVAL, "out is NULL");
    *out = nullptr;
    if (!cfg) return set_error(AV_EINVAL, "cfg is NULL");
    const av_search_config &c = *cfg;
    if (c.num_actions != 4 && c.num_actions != 5)
        return set_error(AV_EINVAL, "num_actions must be 4 or 5");
    if (c.max_frontier < 1 || c.max_frontier > (1 << 24))
        return set_error(AV_EINVAL, "max_frontier must be in [1, 2^24]");
    if (c.table_log2 < 4 || c.table_log2 > 31)
        return set_error(AV_EINVAL, "table_log2 must be in [4, 31]");
    if (c.best_first_k < 0 || c.best_first_k > 512)
        return set_error(AV_EINVAL, "best_first_k must be in [0, 512]");
    if (c.best_first_k > 0 && (c.max_nodes < 1 || c.max_nodes > (1 << 26)))
        return set_error(AV_EINVAL, "max_nodes must be in [1, 2^26]");
    if (c.hash_bits < 0 || c.hash_bits > 63)
        return set_error(AV_EINVAL, "hash_bits must be in [0, 63]");
    const int fcap = c.best_first_k > 0 ? c.best_first_k : c.max_frontier;   // parents per level
    av_config bc{};
    bc.num_envs = c.num_actions * fcap;
    bc.height = c.height; bc.width = c.width; bc.channels = c.channels;
    bc.max_rules = c.max_rules; bc.max_pat_h = c.max_pat_h; bc.max_pat_w = c.max_pat_w;
    bc.per_env_rules = 0; bc.max_episode_steps = c.max_episode_steps;
    bc.device = c.device; bc.engine = c.engine; bc.rule_mode = c.rule_mode; bc.stream = c.stream;
    av_batch_t kids = nullptr;
    if (av_status st = av_create_batch(&bc, &kids)) return st;   // checks the shared limits
    av_search_s *s = new (std::nothrow) av_search_s;
    if (!s) {
        av_destroy_batch(kids);
        return set_error(AV_ENOMEM, "host allocation failed");
    }
    s->cfg = c;
    s->stream = static_cast<hipStream_t>(c.stream);
    s->kids = kids;
    s->row_bytes = batch_row_bytes(kids);
    s->A = c.num_actions;
    s->cap = fcap;
    s->K = c.best_first_k;
    s->slots = uint64_t(1) << c.table_log2;
    const size_t nk = size_t(s->A) * s->cap;
    const size_t fbytes = size_t(c.channels) * s->cap * c.height * s->row_bytes;
    hipError_t e = hipSuccess;
    for (int k = 0; k < 2 && e == hipSuccess; ++k) {
        e = hipMalloc(&s->front[k], fbytes);
        if (e == hipSuccess) e = alloc(&s->reward[k], s->cap);
        if (e == hipSuccess) e = alloc(&s->depth[k], s->cap);
    }
    if (e == hipSuccess) e = alloc(&s->actions, nk);
    if (e == hipSuccess) e = alloc(&s->rew, nk);
    if (e == hipSuccess) e = alloc(&s->done, nk);
    if (e == hipSuccess) e = alloc(&s->kid_reward, nk);
    if (e == hipSuccess) e = alloc(&s->kid_depth, nk);
    if (e == hipSuccess) e = alloc(&s->kid_val, nk);
    if (e == hipSuccess) e = alloc(&s->slot, nk);
    if (e == hipSuccess) e = alloc(&s->block_count, (nk + 255) / 256);
    if (e == hipSuccess) e = alloc(&s->src_of, nk);      // survivors of one level: <= children
    if (e == hipSuccess) e = alloc(&s->keys, s->slots);
    if (e == hipSuccess) e = alloc(&s->vals, s->slots);
    if (e == hipSuccess) e = alloc(&s->claim, s->slots);
    if (e == hipSuccess) e = alloc(&s->epoch, s->slots);
    if (e == hipSuccess)
        e = hipMalloc(&s->store, s->slots * size_t(c.channels) * c.height * s->row_bytes);
    if (e == hipSuccess) e = alloc(&s->best, 1);
    if (e == hipSuccess) e = alloc(&s->counts, 3);
    if (e == hipSuccess && s->K > 0) {
        s->pcap = c.max_nodes;
        const size_t pbytes = size_t(c.channels) * s->pcap * c.height * s->row_bytes;
        e = hipMalloc(&s->pool, pbytes);
        if (e == hipSuccess) e = alloc(&s->pool_reward, s->pcap);
        if (e == hipSuccess) e = alloc(&s->pool_depth, s->pcap);
        if (e == hipSuccess) e = alloc(&s->pool_val, s->pcap);
        if (e == hipSuccess) e = alloc(&s->pool_slot, s->pcap);
        for (int k = 0; k < 2 && e == hipSuccess; ++k) {
            e = alloc(&s->okeys[k], s->pcap);
            if (e == hipSuccess) e = alloc(&s->oids[k], s->pcap);
        }
        if (e == hipSuccess) e = alloc(&s->new_keys, nk);
        if (e == hipSuccess) e = alloc(&s->new_ids, nk);
        if (e == hipSuccess) e = alloc(&s->parents, 512);
        if (e == hipSuccess) e = alloc(&s->n_par, 1);
    }
    if (e == hipSuccess) {
        std::vector<uint8_t> acts(nk);
        for (size_t i = 0; i < nk; ++i) acts[i] = uint8_t(i % s->A + (s->A == 4 ? 1 : 0));
        e = hipMemcpy(s->actions, acts.data(), nk, hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) {
        release(s);
        delete s;
        char m[160];
        std::snprintf(m, sizeof m, "search allocation: %s", hipGetErrorString(e));
        return set_error(e == hipErrorOutOfMemory ? AV_ENOMEM : AV_EDEVICE, m);
    }
    *out = s;
    return AV_OK;
}

av_status av_search_load_rules(av_search_t s, int32_t num_rules, const int32_t *shape,
                               const int8_t *in_pat, const int8_t *out_pat,
                               const int32_t *reward) {
    if (!s) return set_error(AV_EINVAL, "search handle is NULL");
    if (av_status st = av_load_rules(s->kids, num_rules, shape, in_pat, out_pat, reward)) return st;
    s->have_rules = true;
    return AV_OK;
}

av_status av_search_begin(av_search_t s, const uint8_t *root) {
    if (!s) return set_error(AV_EINVAL, "search handle is NULL");
    if (!root) return set_error(AV_EINVAL, "root is NULL");
    if (!s->have_rules) return set_error(AV_ESTATE, "call av_search_load_rules first");
    const av_search_config &c = s->cfg;
    SEARCH_HIP(hipSetDevice(c.device));
    s->cur = 0;
    SEARCH_HIP(launch_pack(root, s->front[0], nullptr, 1, c.channels, c.height, c.width,
                           s->row_bytes, s->stream));
    SEARCH_HIP(hipMemsetAsync(s->reward[0], 0, sizeof(int32_t), s->stream));
    SEARCH_HIP(hipMemsetAsync(s->depth[0], 0, sizeof(int32_t), s->stream));
    SEARCH_HIP(hipMemsetAsync(s->keys, 0, s->slots * sizeof(uint64_t), s->stream));
    SEARCH_HIP(hipMemsetAsync(s->vals, 0, s->slots * sizeof(uint64_t), s->stream));
    SEARCH_HIP(hipMemsetAsync(s->claim, 0, s->slots * sizeof(uint64_t), s->stream));
    SEARCH_HIP(hipMemsetAsync(s->epoch, 0, s->slots * sizeof(uint32_t), s->stream));
    SEARCH_HIP(hipMemsetAsync(s->counts, 0, 3 * sizeof(uint32_t), s->stream));
    SearchArgs a = level_args(s, 1);
    if (s->K > 0) a.root_slot = s->pool_slot;            // the root is pool node 0
    SEARCH_HIP(launch_search_phase(a, s->row_bytes, s->front[0], 1, nullptr, nullptr, s->stream, 3,
                                   0));
    if (s->K > 0) {
        const uint64_t v0 = (uint64_t(0x80000000u) << 32) | 0xFFFFFFFFull;   // (reward 0, depth 0)
        SEARCH_HIP(hipMemsetAsync(s->parents, 0, sizeof(int32_t), s->stream));
        SEARCH_HIP(launch_copy_rows(s->row_bytes, s->front[0], 1, s->parents, s->pool, int(s->pcap),
                                    0, 1, c.channels, c.height, s->stream));
        SEARCH_HIP(hipMemsetAsync(s->pool_reward, 0, sizeof(int32_t), s->stream));
        SEARCH_HIP(hipMemsetAsync(s->pool_depth, 0, sizeof(int32_t), s->stream));
        SEARCH_HIP(hipMemcpyAsync(s->pool_val, &v0, sizeof v0, hipMemcpyHostToDevice, s->stream));
        SEARCH_HIP(hipMemcpyAsync(s->okeys[0], &v0, sizeof v0, hipMemcpyHostToDevice, s->stream));
        SEARCH_HIP(hipMemsetAsync(s->oids[0], 0, sizeof(uint32_t), s->stream));
        SEARCH_HIP(hipStreamSynchronize(s->stream));      // v0 lives on this stack frame
        s->ocur = 0;
        s->pool_n = 1;
        s->open_n = 1;
    }
    s->n_front = 1;
    s->level = 0;
    s->visited = 0;
    s->begun = true;
    return AV_OK;
}

namespace {

// One iteration of batched best-first (av_search_expand with best_first_k > 0).
av_status expand_best_first(av_search_t s, int64_t max_children, av_search_info *info) {
    const av_search_config &c = s->cfg;
    info->parents = 0;
    const int kp = int(std::min<int64_t>(s->K, s->open_n));
    if (kp == 0 || max_children == 0) {
        info->level = s->level;
        info->frontier = s->open_n;
        info->visited = s->visited;
        return read_best(s, info);
    }
    uint32_t npar = 0;
    SEARCH_HIP(launch_bf_pop(s->oids[s->ocur], kp, s->pool_slot, s->pool_val, s->vals, s->parents,
                             s->n_par, s->counts, s->stream));
    SEARCH_HIP(hipMemcpyAsync(&npar, s->n_par, sizeof npar, hipMemcpyDeviceToHost, s->stream));
    SEARCH_HIP(hipStreamSynchronize(s->stream));
    const int64_t n = std::min<int64_t>(int64_t(s->A) * npar, max_children);
    if (s->visited + n > int64_t(0xFFFFFFFEll))
        return set_error(AV_EINVAL, "a search may visit at most 2^32 - 2 states");
    int64_t nn = 0;
    uint32_t counts[3] = {0, 0, 0};
    uint64_t best = 0;                 // read with the counts: final once the children are posted
    if (n > 0) {
        s->cur = 0;
        SEARCH_HIP(launch_copy_rows(s->row_bytes, s->pool, int(s->pcap), s->parents, s->front[0],
                                    int(npar), 0, int(npar), c.channels, c.height, s->stream));
        SEARCH_HIP(launch_bf_gather_meta(s->parents, int(npar), s->pool_reward, s->pool_depth,
                                         s->reward[0], s->depth[0], s->stream));
        SearchArgs a = level_args(s, int(n));
        a.cap = int(s->pcap - s->pool_n);
        a.next_reward = s->pool_reward + s->pool_n;
        a.next_depth = s->pool_depth + s->pool_n;
        void *kst = batch_state(s->kids);           // (bf_pop cleared the counts)
        if (batch_engine(s->kids) == AV_ENGINE_LANE16) {
            if (av_status st = step_prefix(s->kids, int(n), s->actions, s->rew, s->done,
                                           s->front[0], int(npar), s->A, s->depth[0]))
                return st;
        } else {
            SEARCH_HIP(launch_search_phase(a, s->row_bytes, s->front[0], int(npar), kst,
                                           batch_counters(s->kids), s->stream, 0, 0));
            if (av_status st = step_prefix(s->kids, int(n), s->actions, s->rew, s->done)) return st;
        }
        SEARCH_HIP(launch_search_phase(a, s->row_bytes, s->front[0], int(npar), kst, nullptr,
                                       s->stream, 1, 0));
        SEARCH_HIP(hipMemcpyAsync(counts, s->counts, sizeof counts, hipMemcpyDeviceToHost,
                                  s->stream));
        SEARCH_HIP(hipMemcpyAsync(&best, s->best, sizeof best, hipMemcpyDeviceToHost, s->stream));
        SEARCH_HIP(hipStreamSynchronize(s->stream));
        if (counts[1] || int64_t(counts[2]) > s->pcap - s->pool_n) {
            s->begun = false;
            return set_error(AV_ENOMEM, counts[1]
                                            ? "search table too full (an insertion probed 4096 "
                                              "slots); use a larger table_log2 and call "
                                              "av_search_begin again"
                                            : "best-first node pool full; use a larger max_nodes "
                                              "and call av_search_begin again");
        }
        nn = counts[2];
        SEARCH_HIP(launch_copy_rows(s->row_bytes, kst, int(n), s->src_of, s->pool, int(s->pcap),
                                    int(s->pool_n), int(nn), c.channels, c.height, s->stream));
        SEARCH_HIP(launch_bf_append(s->src_of, int(nn), int(s->pool_n), s->kid_val, s->slot,
                                    s->pool_val, s->pool_slot, s->new_keys, s->new_ids,
                                    s->stream));
        s->pool_n += nn;
    }
    const int64_t m = s->open_n - kp;
    SEARCH_HIP(launch_bf_merge(s->okeys[s->ocur] + kp, s->oids[s->ocur] + kp, int(m), s->new_keys,
                               s->new_ids, int(nn), s->okeys[1 - s->ocur], s->oids[1 - s->ocur],
                               s->stream));
    s->ocur = 1 - s->ocur;
    s->open_n = m + nn;
    s->visited += n;
    s->level += 1;
    info->parents = npar;
    info->children = n;
    info->terminal = counts[0];
    info->survivors = nn;
    info->level = s->level;
    info->frontier = s->open_n;
    info->visited = s->visited;
    return n > 0 ? decode_best(best, info) : read_best(s, info);
}

}  // namespace

av_status av_search_expand(av_search_t s, int64_t max_children, av_search_info *info) {
    if (!s) return set_error(AV_EINVAL, "search handle is NULL");
    if (!info) return set_error(AV_EINVAL, "info is NULL");
    if (max_children < 0) return set_error(AV_EINVAL, "max_children must be >= 0");
    if (!s->begun) return set_error(AV_ESTATE, "call av_search_begin first");
    SEARCH_HIP(hipSetDevice(s->cfg.device));
    *info = av_search_info{};
    if (s->K > 0) return expand_best_first(s, max_children, info);
    info->parents = s->n_front;
    const int64_t n = std::min<int64_t>(int64_t(s->A) * s->n_front, max_children);
    uint64_t best = 0;                 // read with the counts: final once the children are posted
    if (s->visited + n > int64_t(0xFFFFFFFEll))
        return set_error(AV_EINVAL, "a search may visit at most 2^32 - 2 states");
    if (n > 0) {
        const av_search_config &c = s->cfg;
        SearchArgs a = level_args(s, int(n));
        void *kst = batch_state(s->kids);
        SEARCH_HIP(hipMemsetAsync(s->counts, 0, 3 * sizeof(uint32_t), s->stream));
        if (batch_engine(s->kids) == AV_ENGINE_LANE16) {
            // the lane16 step reads each child's parent rows and depth itself
            if (av_status st = step_prefix(s->kids, int(n), s->actions, s->rew, s->done,
                                           s->front[s->cur], int(s->n_front), s->A,
                                           s->depth[s->cur]))
                return st;
        } else {
            SEARCH_HIP(launch_search_phase(a, s->row_bytes, s->front[s->cur], int(s->n_front), kst,
                                           batch_counters(s->kids), s->stream, 0, 0));
            if (av_status st = step_prefix(s->kids, int(n), s->actions, s->rew, s->done)) return st;
        }
        SEARCH_HIP(launch_search_phase(a, s->row_bytes, s->front[s->cur], int(s->n_front), kst,
                                       nullptr, s->stream, 1, 0));
        uint32_t counts[3];
        SEARCH_HIP(hipMemcpyAsync(counts, s->counts, sizeof counts, hipMemcpyDeviceToHost,
                                  s->stream));
        SEARCH_HIP(hipMemcpyAsync(&best, s->best, sizeof best, hipMemcpyDeviceToHost, s->stream));
        SEARCH_HIP(hipStreamSynchronize(s->stream));
        if (counts[1]) {
            s->begun = false;
            return set_error(AV_ENOMEM, "search table too full (an insertion probed 4096 slots); "
                                        "use a larger table_log2 and call av_search_begin again");
        }
        const int64_t nn = std::min<int64_t>(counts[2], s->cap);
        a.next_n = int(nn);
        a.next_off = 0;
        SEARCH_HIP(launch_search_phase(a, s->row_bytes, s->front[s->cur], int(s->n_front), kst,
                                       nullptr, s->stream, 2, int(nn)));
        s->cur = 1 - s->cur;
        s->n_front = nn;
        s->visited += n;
        s->level += 1;
        info->children = n;
        info->terminal = counts[0];
        info->survivors = counts[2];
        (void)c;
    }
    info->level = s->level;
    info->frontier = s->n_front;
    info->visited = s->visited;
    return n > 0 ? decode_best(best, info) : read_best(s, info);
}

av_status av_search_frontier(av_search_t s, uint8_t *maps, int32_t *reward, int32_t *depth) {
    if (!s) return set_error(AV_EINVAL, "search handle is NULL");
    if (!s->begun) return set_error(AV_ESTATE, "call av_search_begin first");
    const av_search_config &c = s->cfg;
    SEARCH_HIP(hipSetDevice(c.device));
    if (s->K > 0) {
        SEARCH_HIP(launch_bf_open(s->row_bytes, s->pool, int(s->pcap), s->oids[s->ocur],
                                  int(s->open_n), c.channels, c.height, c.width, maps,
                                  s->pool_reward, s->pool_depth, reward, depth, s->stream));
        return AV_OK;
    }
    const int n = int(s->n_front);
    if (n == 0) return AV_OK;
    if (maps)
        SEARCH_HIP(launch_unpack(s->front[s->cur], maps, n, c.channels, c.height, c.width,
                                 s->row_bytes, s->stream));
    if (reward)
        SEARCH_HIP(hipMemcpyAsync(reward, s->reward[s->cur], n * sizeof(int32_t),
                                  hipMemcpyDeviceToDevice, s->stream));
    if (depth)
        SEARCH_HIP(hipMemcpyAsync(depth, s->depth[s->cur], n * sizeof(int32_t),
                                  hipMemcpyDeviceToDevice, s->stream));
    return AV_OK;
}

av_status av_search_destroy(av_search_t s) {
    if (!s) return AV_OK;
    if (hipSetDevice(s->cfg.device) == hipSuccess) (void)hipStreamSynchronize(s->stream);
    release(s);
    delete s;
    return AV_OK;
}

}  // extern "C"
