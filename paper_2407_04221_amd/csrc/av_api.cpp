// libautoverse host library: the C ABI of include/autoverse.h.
//
// Responsibilities: argument checks (all before any device work), rule compilation into
// the kernels' programs, ownership of the packed device state, kernel-family choice and
// launches on the batch's stream.  Device failures are reported as AV_EDEVICE with the
// HIP error string.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <numeric>
#include <queue>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "av_internal.h"
#include "lane16.h"

using namespace av;

namespace {

thread_local std::string g_last_error;

av_status fail(av_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

#define AV_HIP(call)                                                                  \
    do {                                                                              \
        hipError_t e_ = (call);                                                       \
        if (e_ != hipSuccess)                                                         \
            return fail(AV_EDEVICE, "%s failed: %s", #call, hipGetErrorString(e_));  \
    } while (0)

constexpr char kBlobMagic[8] = {'A', 'V', 'S', 'T', 'A', 'T', 'E', '2'};

struct BlobHeader {
    char magic[8];
    int32_t B, H, W, C, row_bytes, reserved;
    uint64_t state_bytes;
    uint64_t step_no;
};

}  // namespace

struct av_batch_s {
    av_config cfg{};
    hipStream_t stream = nullptr;
    int row_bytes = 0;
    size_t state_bytes = 0;
    void *d_state = nullptr;
    void *d_init = nullptr;
    int32_t *d_t = nullptr;
    uint64_t *d_n = nullptr;         // batch step numbers, one copy per launch unit (B + 8)
    int envs_per_block = 1;
    int engine = AV_ENGINE_GENERIC;   // engine used by the next step
    int plain_engine = AV_ENGINE_GENERIC;   // engine without rule application control
    bool have_rules = false, have_maps = false;
    CtlArgs ctl;                     // rule application control (device arrays owned)
    int32_t R = 0;
    std::vector<uint8_t> features;   // binary rule features, [S][R][2][2][C+1][mh][mw]
    GenericProgram prog;
    DeviceProgram dprog;
    Lane16Program lprog;           // compiled form for the lane16 engine (when chosen)
    Lane16Device dlprog;
    std::vector<std::vector<Lane16Rule>> lsets;   // the rule list the lane16 programs come from
    RowsProgram rprog;             // compiled form for the rows engine (when chosen)
    uint32_t *d_rows = nullptr;
    Lane16Program lprog_ctl;       // lane16 program with rule application control compiled in
    Lane16Device dlprog_ctl;
    bool lane16_ctl = false;       // steps use dlprog_ctl
    // group engine: which environment each workgroup steps, and the cycles each environment
    // took in a launch (device arrays; host copies in pinned memory, filled after launches)
    int32_t *d_order = nullptr;
    uint32_t *d_cost = nullptr;
    int32_t *h_order = nullptr;
    uint32_t *h_cost = nullptr;
    hipEvent_t cost_ev = nullptr;  // recorded after the copy of d_cost to h_cost
    bool cost_pending = false;     // that copy is queued and its costs not used yet
    int simds = 0;                 // SIMDs of the device
};

namespace {

void dev_free(void *p) {
    if (p) (void)hipFree(p);
}

void free_device_program(av_batch_t b) {
    dev_free(b->dprog.hdr);
    dev_free(b->dprog.votes);
    dev_free(b->dprog.match);
    dev_free(b->dprog.vote);
    dev_free(b->dprog.rvote);
    dev_free(b->dprog.gtab);
    dev_free(b->dprog.gmatch);
    b->dprog = DeviceProgram{};
    dev_free(b->d_rows);
    b->d_rows = nullptr;
    lane16_free(b->dlprog);
}

void free_control(av_batch_t b) {
    dev_free(const_cast<int32_t *>(b->ctl.limit));
    dev_free(const_cast<uint32_t *>(b->ctl.inhibit));
    b->ctl = CtlArgs{};
    b->engine = b->plain_engine;
    b->lane16_ctl = false;
    lane16_free(b->dlprog_ctl);
}

}  // namespace

namespace av {

// Output-kernel entry K_O = O - I; unspecified output: no vote; unspecified input: the
// vote points at the output value (paper Sec. 2.1, transposed-convolution write).
int kout(int in, int out) {
    if (out < 0) return 0;
    if (out == 1) return in == 1 ? 0 : 1;
    return in == 0 ? 0 : -1;
}

// The four built-in moves (paper Sec. 2.1: the player moves onto an adjacent cell that
// holds force and no obstacle, consuming the force; Sec. 2.2.1: walls block): rules 0..3
// are right, left, down, up.  Source cell: player 1 -> 0.  Target cell: force 1 and
// wall 0 -> player 1, force 0.
std::vector<HostRule> move_rules(int C) {
    struct Mv { int n, m, sy, sx, ty, tx; };
    const Mv mv[4] = {{1, 2, 0, 0, 0, 1}, {1, 2, 0, 1, 0, 0}, {2, 1, 0, 0, 1, 0}, {2, 1, 1, 0, 0, 0}};
    std::vector<HostRule> out;
    for (const Mv &q : mv) {
        HostRule r;
        r.n = q.n; r.m = q.m; r.reward = 0;
        r.in.assign(size_t(C + 1) * q.n * q.m, -1);
        r.out.assign(size_t(C + 1) * q.n * q.m, -1);
        auto idx = [&](int c, int i, int j) { return (size_t(c) * q.n + i) * q.m + j; };
        r.in[idx(kChPlayer, q.sy, q.sx)] = 1;
        r.out[idx(kChPlayer, q.sy, q.sx)] = 0;
        r.in[idx(C, q.ty, q.tx)] = 1;
        r.in[idx(kChWall, q.ty, q.tx)] = 0;
        r.out[idx(kChPlayer, q.ty, q.tx)] = 1;
        r.out[idx(C, q.ty, q.tx)] = 0;
        out.push_back(std::move(r));
    }
    return out;
}

// Order in which a rule's input entries are tested: rarest evidence first, so a thread
// can stop as soon as its whole row has failed.  Force and player bits are rare; walls
// and empty tiles are common; a must-be-1 entry rejects more than a must-be-0 one.
int entry_rank(int c, int want, int C) {
    int ch;
    if (c == C) ch = 0;
    else if (c == kChPlayer) ch = 1;
    else if (c == kChGoal || c >= 4) ch = 2;
    else if (c == kChWall) ch = 3;
    else ch = 4;
    return (want ? 0 : 8) + ch;
}

void compile_generic(const std::vector<std::vector<HostRule>> &sets, int C, bool force_votes,
                     GenericProgram &p) {
    const int C1 = C + 1;
    p.any_reward = 0;
    p.sets = int(sets.size());
    p.rules_per_set = int(sets[0].size());
    std::vector<std::vector<uint32_t>> match(sets.size()), vote(sets.size()), rvote(sets.size());
    p.hdr.assign(size_t(p.sets) * p.rules_per_set, RuleHdr{});
    p.votes.assign(size_t(p.sets) * C1, VoteList{});
    for (size_t s = 0; s < sets.size(); ++s) {
        std::vector<std::vector<uint32_t>> per_ch(C1);
        for (int r = 0; r < p.rules_per_set; ++r) {
            const HostRule &hr = sets[s][r];
            RuleHdr &h = p.hdr[s * p.rules_per_set + r];
            h.n = hr.n; h.m = hr.m; h.reward = hr.reward;
            h.match_off = int(match[s].size());
            std::vector<std::pair<int, uint32_t>> ents;
            for (int c = 0; c < C1; ++c)
                for (int i = 0; i < hr.n; ++i)
                    for (int j = 0; j < hr.m; ++j) {
                        const int w = hr.at(hr.in, c, i, j);
                        if (w >= 0) ents.push_back({entry_rank(c, w, C), pack_match(c, i, j, w)});
                        const int k = kout(w, hr.at(hr.out, c, i, j));
                        if (k) per_ch[c].push_back(pack_vote(r, i, j, k > 0));
                    }
            h.vote_off = int(rvote[s].size());
            for (int c = 0; c < (force_votes ? C1 : C); ++c)
                for (int i = 0; i < hr.n; ++i)
                    for (int j = 0; j < hr.m; ++j) {
                        const int k = kout(hr.at(hr.in, c, i, j), hr.at(hr.out, c, i, j));
                        if (k) rvote[s].push_back(pack_vote(c, i, j, k > 0));
                    }
            h.vote_cnt = int(rvote[s].size()) - h.vote_off;
            h.pad = 0;                    // bit c: the rule casts a rule-major vote on channel c
            for (int e = h.vote_off; e < int(rvote[s].size()); ++e)
                if ((rvote[s][e] & 255u) < 32u) h.pad |= int32_t(1u << (rvote[s][e] & 255u));
            if (hr.reward != 0) p.any_reward = 1;
            std::stable_sort(ents.begin(), ents.end(),
                             [](auto &a, auto &b) { return a.first < b.first; });
            for (auto &e : ents) match[s].push_back(e.second);
            h.match_cnt = int(match[s].size()) - h.match_off;
        }
        for (int c = 0; c < C1; ++c) {
            p.votes[s * C1 + c] = VoteList{int(vote[s].size()), int(per_ch[c].size())};
            vote[s].insert(vote[s].end(), per_ch[c].begin(), per_ch[c].end());
        }
    }
    p.match_stride = 1;
    p.vote_stride = 1;
    p.rvote_stride = 1;
    for (size_t s = 0; s < sets.size(); ++s) {
        p.match_stride = std::max(p.match_stride, int(match[s].size()));
        p.vote_stride = std::max(p.vote_stride, int(vote[s].size()));
        p.rvote_stride = std::max(p.rvote_stride, int(rvote[s].size()));
    }
    p.rvote.assign(size_t(p.sets) * p.rvote_stride, 0);
    for (size_t s = 0; s < sets.size(); ++s)
        std::copy(rvote[s].begin(), rvote[s].end(), p.rvote.begin() + s * p.rvote_stride);
    p.match.assign(size_t(p.sets) * p.match_stride, 0);
    p.vote.assign(size_t(p.sets) * p.vote_stride, 0);
    for (size_t s = 0; s < sets.size(); ++s) {
        std::copy(match[s].begin(), match[s].end(), p.match.begin() + s * p.match_stride);
        std::copy(vote[s].begin(), vote[s].end(), p.vote.begin() + s * p.vote_stride);
    }
}


// The moves followed by each set's loaded rules, checked (shapes within the map and the
// pattern array, values in {-1, 0, 1}, an exact float reward): the rule sets of
// av_load_rules' arguments (paper Sec. 2.1: rules are n x m input and output patterns with a
// reward).
av_status parse_rule_sets(const av_config &c, int32_t R, const int32_t *shape,
                          const int8_t *in_pat, const int8_t *out_pat, const int32_t *reward,
                          std::vector<std::vector<HostRule>> &sets) {
    const int S = c.per_env_rules ? c.num_envs : 1;
    const int C1 = c.channels + 1, ph = c.max_pat_h, pw = c.max_pat_w;
    const size_t pat = size_t(C1) * ph * pw;
    sets.assign(S, {});
    const std::vector<HostRule> moves = move_rules(c.channels);
    for (int s = 0; s < S; ++s) {
        sets[s] = moves;
        long long worst = 0;
        for (int r = 0; r < R; ++r) {
            const size_t k = size_t(s) * R + r;
            HostRule hr;
            hr.n = shape[2 * k];
            hr.m = shape[2 * k + 1];
            hr.reward = reward[k];
            if (hr.n < 1 || hr.n > ph || hr.n > c.height || hr.m < 1 || hr.m > pw || hr.m > c.width)
                return fail(AV_EINVAL, "set %d rule %d: shape %d x %d outside [1, min(max_pat, map)]",
                            s, r, hr.n, hr.m);
            for (size_t e = 0; e < pat; ++e) {
                const int vi = in_pat[k * pat + e], vo = out_pat[k * pat + e];
                if (vi < -1 || vi > 1 || vo < -1 || vo > 1)
                    return fail(AV_EINVAL, "set %d rule %d: pattern value outside {-1, 0, 1}", s, r);
            }
            hr.in.assign(size_t(C1) * hr.n * hr.m, -1);
            hr.out.assign(size_t(C1) * hr.n * hr.m, -1);
            for (int ch = 0; ch < C1; ++ch)
                for (int i = 0; i < hr.n; ++i)
                    for (int j = 0; j < hr.m; ++j) {
                        const size_t src = k * pat + (size_t(ch) * ph + i) * pw + j;
                        hr.in[(size_t(ch) * hr.n + i) * hr.m + j] = in_pat[src];
                        hr.out[(size_t(ch) * hr.n + i) * hr.m + j] = out_pat[src];
                    }
            const long long rw = hr.reward < 0 ? -(long long)hr.reward : hr.reward;
            worst += rw * (long long)(c.height - hr.n + 1) * (c.width - hr.m + 1);
            sets[s].push_back(std::move(hr));
        }
        if (worst >= (1LL << 24))
            return fail(AV_EINVAL, "set %d: |reward| x anchors sums to %lld >= 2^24; the float "
                        "reward would not be exact", s, worst);
    }
    return AV_OK;
}

}  // namespace av

namespace {

template <typename T>
av_status upload(T **dst, const std::vector<T> &src) {
    const size_t n = std::max<size_t>(src.size(), 1) * sizeof(T);
    AV_HIP(hipMalloc(reinterpret_cast<void **>(dst), n));
    if (!src.empty()) AV_HIP(hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice));
    return AV_OK;
}

// The group engine's order and cost arrays, once per batch: workgroup i starts on
// environment i; a step reorders them (group_order_update).
av_status group_order_init(av_batch_t b) {
    const int B = b->cfg.num_envs;
    if (b->d_order) {
        b->cost_pending = false;                  // costs of another rule set
        std::iota(b->h_order, b->h_order + B, 0);
        AV_HIP(hipMemcpy(b->d_order, b->h_order, sizeof(int32_t) * size_t(B), hipMemcpyHostToDevice));
        return AV_OK;
    }
    int cus = 0;
    AV_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, b->cfg.device));
    b->simds = 4 * cus;                           // 4 SIMDs per CU
    AV_HIP(hipHostMalloc(reinterpret_cast<void **>(&b->h_order), sizeof(int32_t) * size_t(B)));
    AV_HIP(hipHostMalloc(reinterpret_cast<void **>(&b->h_cost), sizeof(uint32_t) * size_t(B)));
    AV_HIP(hipEventCreateWithFlags(&b->cost_ev, hipEventDisableTiming));
    std::vector<int32_t> ident(static_cast<size_t>(B));
    std::iota(ident.begin(), ident.end(), 0);
    std::copy(ident.begin(), ident.end(), b->h_order);
    if (av_status st = upload(&b->d_order, ident)) return st;
    return upload(&b->d_cost, std::vector<uint32_t>(size_t(B), 0u));
}

// Copies of the batch step number: one per launch unit (at most one per environment, and
// the lane16 engine's last workgroup may hold up to three waves past the batch), plus slack.
int step_copies(int B) { return B + 8; }

av_status check_batch(av_batch_t b) {
    if (!b) return fail(AV_EINVAL, "batch handle is NULL");
    return AV_OK;
}

av_status set_device(av_batch_t b) {
    AV_HIP(hipSetDevice(b->cfg.device));
    return AV_OK;
}

}  // namespace

namespace av {

void *batch_state(av_batch_t b) { return b->d_state; }
int32_t *batch_counters(av_batch_t b) { return b->d_t; }
int batch_row_bytes(av_batch_t b) { return b->row_bytes; }
av_status set_error(av_status st, const char *msg) { return fail(st, "%s", msg); }

int batch_engine(av_batch_t b) { return b->engine; }

av_status step_prefix(av_batch_t b, int n, const uint8_t *actions, float *rewards,
                      uint8_t *done, const void *gsrc, int gnf, int gA, const int32_t *gdepth) {
    const av_config &c = b->cfg;
    if (n < 1 || n > c.num_envs) return fail(AV_EINVAL, "prefix of %d environments", n);
    if (!b->have_rules) return fail(AV_ESTATE, "no rules loaded");
    StepArgs a{};
    a.B = n; a.H = c.height; a.W = c.width; a.C = c.channels;
    a.L = c.max_episode_steps; a.per_env = 0; a.k = 1;
    a.sequential = c.rule_mode == AV_RULES_SEQUENTIAL;
    a.row_bytes = b->row_bytes; a.max_pat_h = c.max_pat_h;
    a.max_pat_w = c.max_pat_w;
    a.state = b->d_state; a.init = b->d_init; a.t = b->d_t; a.nctr = b->d_n;
    a.actions = actions; a.rewards = rewards; a.done = done;
    a.prog = b->dprog;
    if (gsrc && b->engine != AV_ENGINE_LANE16)
        return fail(AV_EINVAL, "gathering step on a non-lane16 batch");
    a.gsrc = gsrc; a.gnf = gnf; a.gA = gA; a.gdepth = gdepth;
    if (b->engine == AV_ENGINE_LANE16)
        AV_HIP(launch_lane16_step(a, b->dlprog, b->stream));
    else if (b->engine == AV_ENGINE_ROWS)
        AV_HIP(launch_rows_step(a, b->d_rows, b->rprog.set_words, b->rprog.rules, b->stream));
    else if (b->engine == AV_ENGINE_WAVE)
        AV_HIP(launch_wave_step(a, b->stream));
    else if (b->engine == AV_ENGINE_GROUP)
        AV_HIP(launch_group_step(a, b->stream));
    else
        AV_HIP(launch_generic_step(a, b->envs_per_block, b->stream));
    return AV_OK;
}

}  // namespace av

extern "C" {

const char *av_last_error(void) { return g_last_error.c_str(); }

av_status av_create_batch(const av_config *cfg, av_batch_t *out) {
    g_last_error.clear();
    if (!out) return fail(AV_EINVAL, "out is NULL");
    *out = nullptr;
    if (!cfg) return fail(AV_EINVAL, "cfg is NULL");
    const av_config &c = *cfg;
    if (c.num_envs < 1) return fail(AV_EINVAL, "num_envs must be >= 1 (got %d)", c.num_envs);
    if (c.height < 1 || c.height > kMaxDim || c.width < 1 || c.width > kMaxDim)
        return fail(AV_EINVAL, "height and width must be in [1, %d] (got %d x %d)", kMaxDim,
                    c.height, c.width);
    if (c.channels < 4 || c.channels > 31)
        return fail(AV_EINVAL, "channels must be in [4, 31] (got %d)", c.channels);
    if (c.max_rules < 0 || c.max_rules > kMaxRules)
        return fail(AV_EINVAL, "max_rules must be in [0, %d] (got %d)", kMaxRules, c.max_rules);
    if (c.max_pat_h < 1 || c.max_pat_h > kMaxPat || c.max_pat_w < 1 || c.max_pat_w > kMaxPat)
        return fail(AV_EINVAL, "max_pat_h and max_pat_w must be in [1, %d]", kMaxPat);
    if (c.per_env_rules != 0 && c.per_env_rules != 1)
        return fail(AV_EINVAL, "per_env_rules must be 0 or 1");
    if (c.max_episode_steps < 0) return fail(AV_EINVAL, "max_episode_steps must be >= 0");
    if (c.rule_mode != AV_RULES_PARALLEL && c.rule_mode != AV_RULES_SEQUENTIAL)
        return fail(AV_EINVAL, "unknown rule_mode %d", c.rule_mode);
    if (c.engine < AV_ENGINE_AUTO || c.engine > AV_ENGINE_GROUP)
        return fail(AV_EINVAL, "unknown engine %d", c.engine);
    const size_t env_lds = generic_env_lds_bytes(c.height, c.width, c.channels,
                                                 c.max_rules + kMoveRules);
    if (env_lds > size_t(kLdsBudget))
        return fail(AV_EINVAL, "one environment needs %zu bytes of LDS (limit %d): fewer rules, "
                    "channels or a smaller map", env_lds, kLdsBudget);
    const bool lane16_ok = lane16_eligible(c);
    if (c.engine == AV_ENGINE_LANE16 && !lane16_ok)
        return fail(AV_EINVAL, "the lane16 engine needs H, W <= 16 and one rule set shared by "
                    "all environments");
    const size_t wave_lds = wave_lds_bytes(c.height, c.width, c.channels, c.max_rules + kMoveRules);
    const bool wave_ok = wave_lds <= size_t(kLdsBudget);
    if (c.engine == AV_ENGINE_WAVE && !wave_ok)
        return fail(AV_EINVAL, "the wave engine needs %zu bytes of LDS (limit %d)", wave_lds,
                    kLdsBudget);
    const bool group_ok = c.rule_mode == AV_RULES_PARALLEL &&
                          group_eligible(c.height, c.width, c.channels, c.max_rules + kMoveRules,
                                         c.max_pat_h, c.max_pat_w);
    if (c.engine == AV_ENGINE_GROUP && !group_ok)
        return fail(AV_EINVAL, "the group engine needs parallel rule order, H, W <= 32, "
                    "(max_rules + 4) x max_pat_h x max_pat_w <= 254 and a working set within "
                    "64 KiB of LDS");
    const bool rows_ok = rows_eligible(c.height, c.width, c.channels, c.max_rules + kMoveRules);
    if (c.engine == AV_ENGINE_ROWS && !rows_ok)
        return fail(AV_EINVAL, "the rows engine needs at most 60 rules and %zu bytes of LDS (limit %d)",
                    rows_lds_bytes(c.height, c.width, c.channels, c.max_rules + kMoveRules), kLdsBudget);

    int dev_count = 0;
    AV_HIP(hipGetDeviceCount(&dev_count));
    if (c.device < 0 || c.device >= dev_count)
        return fail(AV_EINVAL, "device %d out of range (%d devices)", c.device, dev_count);
    AV_HIP(hipSetDevice(c.device));

    av_batch_s *b = new (std::nothrow) av_batch_s;
    if (!b) return fail(AV_ENOMEM, "host allocation failed");
    b->cfg = c;
    b->stream = static_cast<hipStream_t>(c.stream);
    b->row_bytes = c.width <= 16 ? 2 : (c.width <= 32 ? 4 : 8);
    b->state_bytes = size_t(c.channels) * c.num_envs * c.height * b->row_bytes;
    b->envs_per_block = std::max(1, std::min(256 / c.height, int(kLdsBudget / env_lds)));
    if (c.engine != AV_ENGINE_AUTO) b->engine = c.engine;
    else if (lane16_ok) b->engine = AV_ENGINE_LANE16;
    // measured on MI355X: per-environment rule sets in parallel order run fastest on the group
    // engine (16 x 16, 8 rules: 1.5 / 5.0 / 26 us per step with literal / planted / dense
    // rules against the wave engine's 2.7 / 4.5 / 69; 32 x 32, 16 rules: 11.8 / 24.7 / 113
    // against 17.6 / 31.0 / 228), otherwise on the wave engine (its rule groups match many
    // rules of a crowded environment at once); shared sets the lane16 engine cannot take run
    // on rows (64 x 64, 32 rules: 3.2 against the wave engine's 7.7 us per step)
    else if (c.per_env_rules && group_ok) b->engine = AV_ENGINE_GROUP;
    else if (c.per_env_rules && wave_ok) b->engine = AV_ENGINE_WAVE;
    else if (rows_ok) b->engine = AV_ENGINE_ROWS;
    else b->engine = wave_ok ? AV_ENGINE_WAVE : AV_ENGINE_GENERIC;
    b->plain_engine = b->engine;
    hipError_t e = hipMalloc(&b->d_state, b->state_bytes);
    if (e == hipSuccess) e = hipMalloc(&b->d_init, b->state_bytes);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&b->d_t), sizeof(int32_t) * c.num_envs);
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&b->d_n), sizeof(uint64_t) * step_copies(c.num_envs));
    if (e == hipSuccess) e = hipMemset(b->d_state, 0, b->state_bytes);
    if (e == hipSuccess) e = hipMemset(b->d_init, 0, b->state_bytes);
    if (e == hipSuccess) e = hipMemset(b->d_t, 0, sizeof(int32_t) * c.num_envs);
    if (e == hipSuccess) e = hipMemset(b->d_n, 0, sizeof(uint64_t) * step_copies(c.num_envs));
    if (e != hipSuccess) {
        dev_free(b->d_state); dev_free(b->d_init); dev_free(b->d_t); dev_free(b->d_n);
        delete b;
        return fail(e == hipErrorOutOfMemory ? AV_ENOMEM : AV_EDEVICE, "device allocation: %s",
                    hipGetErrorString(e));
    }
    *out = b;
    return AV_OK;
}

av_status av_load_rules(av_batch_t b, int32_t R, const int32_t *shape, const int8_t *in_pat,
                        const int8_t *out_pat, const int32_t *reward) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    const av_config &c = b->cfg;
    if (R < 0 || R > c.max_rules)
        return fail(AV_EINVAL, "num_rules %d outside [0, max_rules = %d]", R, c.max_rules);
    if (R > 0 && (!shape || !in_pat || !out_pat || !reward))
        return fail(AV_EINVAL, "rule arrays must not be NULL");
    const int S = c.per_env_rules ? c.num_envs : 1;
    const int C1 = c.channels + 1, ph = c.max_pat_h, pw = c.max_pat_w;
    const size_t pat = size_t(C1) * ph * pw;
    std::vector<std::vector<HostRule>> sets;
    if (av_status st = parse_rule_sets(c, R, shape, in_pat, out_pat, reward, sets)) return st;
    std::vector<uint8_t> feats(size_t(S) * R * 4 * pat);
    for (size_t k = 0; k < size_t(S) * R; ++k)
        for (int io = 0; io < 2; ++io) {
            const int8_t *src = (io ? out_pat : in_pat) + k * pat;
            uint8_t *spec = &feats[((k * 2 + io) * 2 + 0) * pat];
            uint8_t *val = &feats[((k * 2 + io) * 2 + 1) * pat];
            for (size_t e = 0; e < pat; ++e) {
                spec[e] = src[e] != -1;
                val[e] = src[e] == 1;
            }
        }
    if (av_status st = set_device(b)) return st;
    AV_HIP(hipStreamSynchronize(b->stream));   // no step may still read the old program
    free_device_program(b);
    free_control(b);
    b->have_rules = false;
    compile_generic(sets, c.channels, c.rule_mode == AV_RULES_SEQUENTIAL, b->prog);
    if (av_status st = upload(&b->dprog.hdr, b->prog.hdr)) return st;
    if (av_status st = upload(&b->dprog.votes, b->prog.votes)) return st;
    if (av_status st = upload(&b->dprog.match, b->prog.match)) return st;
    if (av_status st = upload(&b->dprog.vote, b->prog.vote)) return st;
    if (av_status st = upload(&b->dprog.rvote, b->prog.rvote)) return st;
    b->dprog.rules_per_set = b->prog.rules_per_set;
    b->dprog.match_stride = b->prog.match_stride;
    b->dprog.vote_stride = b->prog.vote_stride;
    b->dprog.rvote_stride = b->prog.rvote_stride;
    b->dprog.any_reward = b->prog.any_reward;
    if (b->plain_engine == AV_ENGINE_GROUP) {
        std::vector<uint32_t> tab;
        std::vector<uint32_t> gm;
        compile_group_tables(b->prog, c.height, c.width, c.channels, c.max_pat_h, tab,
                             b->dprog.gtab_stride, gm, b->dprog.gmatch_stride);
        if (av_status st = upload(&b->dprog.gtab, tab)) return st;
        if (av_status st = upload(&b->dprog.gmatch, gm)) return st;
        if (av_status st = group_order_init(b)) return st;
    }
    if (b->plain_engine == AV_ENGINE_ROWS) {
        compile_rows(b->prog, c.channels, b->rprog);
        if (av_status st = upload(&b->d_rows, b->rprog.words)) return st;
    }
    if (b->engine == AV_ENGINE_LANE16) {
        std::vector<std::vector<Lane16Rule>> lsets(S);
        for (int s = 0; s < S; ++s)
            for (const HostRule &hr : sets[s]) {
                Lane16Rule lr;
                lr.n = hr.n; lr.m = hr.m; lr.reward = hr.reward;
                lr.in = hr.in; lr.out = hr.out;
                lsets[s].push_back(std::move(lr));
            }
        lane16_compile(lsets, c.channels, c.height, c.width, c.max_episode_steps,
                       c.rule_mode == AV_RULES_SEQUENTIAL, b->lprog);
        std::string log;
        hipError_t e = lane16_upload(b->lprog, b->dlprog, &log);
        if (e != hipSuccess)
            return fail(AV_EDEVICE, "lane16 kernel build: %s %s", hipGetErrorString(e), log.c_str());
        b->lsets.swap(lsets);
    }
    b->R = R;
    b->features.swap(feats);
    b->have_rules = true;
    return AV_OK;
}

av_status av_reset(av_batch_t b, const uint8_t *init_maps) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    if (!init_maps) return fail(AV_EINVAL, "init_maps is NULL");
    if (av_status st = set_device(b)) return st;
    const av_config &c = b->cfg;
    AV_HIP(launch_pack(init_maps, b->d_init, b->d_state, c.num_envs, c.channels, c.height, c.width,
                       b->row_bytes, b->stream));
    // step counters and batch step numbers to 0 with a kernel (no memset node under capture)
    AV_HIP(launch_fill_counters(b->d_t, c.num_envs, b->d_n, step_copies(c.num_envs), 0, 0,
                                b->stream));
    b->have_maps = true;
    return AV_OK;
}

av_status av_set_rule_control(av_batch_t b, const int32_t *limit, const uint8_t *inhibit,
                              int32_t order, uint64_t seed) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    if (!b->have_rules) return fail(AV_ESTATE, "call av_load_rules first");
    if (order != AV_SITES_ROW_MAJOR && order != AV_SITES_RANDOM)
        return fail(AV_EINVAL, "unknown site order %d", order);
    const av_config &c = b->cfg;
    const int S = c.per_env_rules ? c.num_envs : 1, R = b->R, Rt = R + kMoveRules;
    bool active = false;
    if (limit)
        for (size_t k = 0; k < size_t(S) * R; ++k) {
            if (limit[k] < 0)
                return fail(AV_EINVAL, "set %zu rule %zu: negative limit %d", k / R, k % R, limit[k]);
            active |= limit[k] > 0;
        }
    if (inhibit)
        for (size_t s = 0; s < size_t(S); ++s)
            for (int q = 0; q < R; ++q)
                for (int r = 0; r < R; ++r)
                    if (inhibit[(s * R + q) * R + r]) {
                        if (q >= r)
                            return fail(AV_EINVAL, "set %zu: rule %d may not inhibit rule %d "
                                        "(only earlier rules inhibit later ones)", s, q, r);
                        active = true;
                    }
    const bool random = order == AV_SITES_RANDOM;
    // control compiles into the lane16 program; the wave engine runs it when its scratch fits
    // in LDS; otherwise it runs on the generic engine
    // (a rows or group batch created with AV_ENGINE_AUTO switches like a wave batch; an
    // explicit rows or group batch has no control)
    const bool on_lane16 = b->plain_engine == AV_ENGINE_LANE16;
    const bool wave_like = b->plain_engine == AV_ENGINE_WAVE ||
                           ((b->plain_engine == AV_ENGINE_ROWS ||
                             b->plain_engine == AV_ENGINE_GROUP) && c.engine == AV_ENGINE_AUTO);
    const bool on_wave = wave_like &&
                         wave_lds_bytes(c.height, c.width, c.channels, R + kMoveRules, true,
                                        random) <= size_t(kLdsBudget);
    if (active && (c.engine == AV_ENGINE_ROWS || c.engine == AV_ENGINE_GROUP))
        return fail(AV_EINVAL, "the %s engine has no rule application control; create the "
                    "batch with AV_ENGINE_AUTO, AV_ENGINE_WAVE or AV_ENGINE_GENERIC",
                    c.engine == AV_ENGINE_ROWS ? "rows" : "group");
    if (active && !on_lane16 && !on_wave && c.engine != AV_ENGINE_AUTO &&
        c.engine != AV_ENGINE_GENERIC)
        return fail(AV_EINVAL, "rule application control does not fit this wave batch's LDS; "
                    "create the batch with AV_ENGINE_AUTO or AV_ENGINE_GENERIC");
    const size_t env_lds = generic_env_lds_bytes(c.height, c.width, c.channels, Rt, true, random);
    if (active && env_lds > size_t(kLdsBudget))
        return fail(AV_EINVAL, "rule application control needs %zu bytes of LDS per environment "
                    "(limit %d)", env_lds, kLdsBudget);
    if (av_status st = set_device(b)) return st;
    AV_HIP(hipStreamSynchronize(b->stream));   // no step may still read the old arrays
    free_control(b);
    // the engine, or its workgroup shape, may change below: every launch unit's copy of the
    // batch step number takes copy 0's value, which every engine keeps current
    AV_HIP(launch_fill_counters(nullptr, 0, b->d_n, step_copies(c.num_envs), 1, 0, b->stream));
    if (!active) return AV_OK;
    const int words = (Rt + 31) / 32;
    std::vector<int32_t> lim(size_t(S) * Rt, 0);
    std::vector<uint32_t> inh(size_t(S) * Rt * words, 0);
    for (size_t s = 0; s < size_t(S); ++s)
        for (int r = 0; r < R; ++r) {
            if (limit) lim[s * Rt + kMoveRules + r] = limit[s * R + r];
            if (inhibit)
                for (int q = 0; q < r; ++q)
                    if (inhibit[(s * R + q) * R + r]) {
                        const int qi = kMoveRules + q;
                        inh[(s * Rt + kMoveRules + r) * words + qi / 32] |= 1u << (qi % 32);
                    }
        }
    int32_t *d_lim = nullptr;
    uint32_t *d_inh = nullptr;
    if (av_status st = upload(&d_lim, lim)) return st;
    b->ctl.limit = d_lim;
    if (av_status st = upload(&d_inh, inh)) { free_control(b); return st; }
    b->ctl.inhibit = d_inh;
    b->ctl.words = words;
    b->ctl.active = 1;
    b->ctl.random = random;
    b->ctl.seed = seed;
    if (on_lane16) {
        Lane16Control lc;
        lc.random = random;
        lc.limit.assign(Rt, 0);
        lc.inhibitors.assign(Rt, {});
        for (int r = 0; r < R; ++r) {
            if (limit) lc.limit[kMoveRules + r] = limit[r];
            if (inhibit)
                for (int q = 0; q < r; ++q)
                    if (inhibit[size_t(q) * R + r]) lc.inhibitors[kMoveRules + r].push_back(kMoveRules + q);
        }
        lane16_compile(b->lsets, c.channels, c.height, c.width, c.max_episode_steps,
                       c.rule_mode == AV_RULES_SEQUENTIAL, b->lprog_ctl, &lc);
        std::string log;
        hipError_t e = lane16_upload(b->lprog_ctl, b->dlprog_ctl, &log);
        if (e != hipSuccess) {
            free_control(b);
            return fail(AV_EDEVICE, "lane16 kernel build: %s %s", hipGetErrorString(e), log.c_str());
        }
        b->lane16_ctl = true;
        b->engine = AV_ENGINE_LANE16;
    } else if (on_wave) {
        b->engine = AV_ENGINE_WAVE;
    } else {
        b->engine = AV_ENGINE_GENERIC;
    }
    return AV_OK;
}

// Group engine: the order in which workgroups take environments.  With several waves per SIMD,
// workgroups i, i + P, i + 2P, ... (P: the device's SIMDs) share a SIMD, and a launch lasts as
// long as its slowest SIMD.  An environment's steps cost about the same from launch to launch
// (its rule set does not change), so, from the cycles each took in an earlier launch of 64
// steps or more, environments are dealt slowest first, each to the SIMD with the least work so
// far among those with a workgroup left (longest processing time first): the P slowest get a
// SIMD each, and the slowest one's SIMD gets the lightest of the rest.  Results do not depend
// on the order.  The
// costs come back through an asynchronous copy; a launch uses them once that copy is done,
// and never while the stream is being captured.
constexpr int kGroupOrderMinSteps = 64;

static bool capturing(hipStream_t s) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    return hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone;
}

static hipError_t group_order_update(av_batch_t b, int k) {
    if (!b->d_order || k < kGroupOrderMinSteps || !b->cost_pending || capturing(b->stream))
        return hipSuccess;
    if (hipEventQuery(b->cost_ev) != hipSuccess) return hipSuccess;   // not back yet
    b->cost_pending = false;
    const int B = b->cfg.num_envs, P = b->simds;
    std::vector<int> idx(static_cast<size_t>(B));
    std::iota(idx.begin(), idx.end(), 0);
    std::stable_sort(idx.begin(), idx.end(),
                     [&](int x, int y) { return b->h_cost[x] > b->h_cost[y]; });
    // SIMD j holds workgroups j, j + P, ...: (work so far, j) of the SIMDs with one left
    std::vector<int> used(static_cast<size_t>(P), 0);
    std::priority_queue<std::pair<uint64_t, int>, std::vector<std::pair<uint64_t, int>>,
                        std::greater<std::pair<uint64_t, int>>> open;
    for (int j = 0; j < P; ++j) open.push({0ull, j});
    for (int e : idx) {
        const auto [work, j] = open.top();
        open.pop();
        const int i = used[size_t(j)]++ * P + j;
        b->h_order[i] = e;
        if (i + P < B) open.push({work + b->h_cost[e], j});
    }
    return hipMemcpyAsync(b->d_order, b->h_order, sizeof(int32_t) * size_t(B),
                          hipMemcpyHostToDevice, b->stream);
}

static hipError_t group_cost_collect(av_batch_t b, int k) {
    // (a batch of at most P environments has one wave per SIMD: nothing to deal)
    if (!b->d_order || k < kGroupOrderMinSteps || b->cost_pending || b->cfg.num_envs <= b->simds ||
        capturing(b->stream))
        return hipSuccess;
    hipError_t e = hipMemcpyAsync(b->h_cost, b->d_cost, sizeof(uint32_t) * size_t(b->cfg.num_envs),
                                  hipMemcpyDeviceToHost, b->stream);
    if (e == hipSuccess) e = hipEventRecord(b->cost_ev, b->stream);
    if (e == hipSuccess) b->cost_pending = true;
    return e;
}

static av_status step_k(av_batch_t b, int32_t k, const uint8_t *actions, float *rewards,
                        uint8_t *done, uint8_t *obs = nullptr, int32_t w = 0) {
    if (av_status st = check_batch(b)) return st;
    if (k < 1) return fail(AV_EINVAL, "k must be >= 1 (got %d)", k);
    if (!actions || !rewards || !done) return fail(AV_EINVAL, "actions, rewards and done must not be NULL");
    if (!b->have_rules || !b->have_maps)
        return fail(AV_ESTATE, "call av_load_rules and av_reset before stepping");
    if (av_status st = set_device(b)) return st;
    const av_config &c = b->cfg;
    StepArgs a{};
    a.B = c.num_envs; a.H = c.height; a.W = c.width; a.C = c.channels;
    a.L = c.max_episode_steps; a.per_env = c.per_env_rules; a.k = k;
    a.sequential = c.rule_mode == AV_RULES_SEQUENTIAL;
    a.row_bytes = b->row_bytes; a.max_pat_h = c.max_pat_h;
    a.max_pat_w = c.max_pat_w;
    a.state = b->d_state; a.init = b->d_init; a.t = b->d_t; a.nctr = b->d_n;
    a.actions = actions; a.rewards = rewards; a.done = done;
    a.prog = b->dprog;
    a.ctl = b->ctl;
    // the lane16 kernel writes small windows itself (one byte per lane and store); larger
    // windows are faster through the observation kernel's 16-byte stores
    // LDS of the fused path: its window buffers, the staged rows (1 KiB per channel) and
    // player cells, and with random-order control the site keys (32 KiB)
    const int fused_lds = 4 * ((8 * c.channels * w * w + 16 + 15) & ~15) + c.channels * 1024 +
                          128 + (b->lane16_ctl && b->ctl.random ? 32 * 1024 : 0);
    const bool fused = obs && b->engine == AV_ENGINE_LANE16 && w <= kFusedObserveMax &&
                       fused_lds <= kLdsBudget;
    if (fused) {
        a.obs = obs;
        a.obs_w = w;
    }
    if (b->engine == AV_ENGINE_LANE16) {
        AV_HIP(launch_lane16_step(a, b->lane16_ctl ? b->dlprog_ctl : b->dlprog, b->stream));
    } else if (b->engine == AV_ENGINE_ROWS) {
        AV_HIP(launch_rows_step(a, b->d_rows, b->rprog.set_words, b->rprog.rules, b->stream));
    } else if (b->engine == AV_ENGINE_GROUP) {
        AV_HIP(group_order_update(b, k));
        a.order = b->d_order;
        a.cost = b->d_cost;
        AV_HIP(launch_group_step(a, b->stream));
        AV_HIP(group_cost_collect(b, k));
    } else if (b->engine == AV_ENGINE_WAVE) {
        AV_HIP(launch_wave_step(a, b->stream));
    } else {
        int G = b->envs_per_block;
        if (a.ctl.active) {
            const size_t env_lds = generic_env_lds_bytes(c.height, c.width, c.channels,
                                                         b->dprog.rules_per_set, true,
                                                         a.ctl.random);
            G = std::max(1, std::min(256 / c.height, int(kLdsBudget / env_lds)));
        }
        AV_HIP(launch_generic_step(a, G, b->stream));
    }
    if (obs && !fused)
        AV_HIP(launch_observe(b->d_state, c.num_envs, c.channels, c.height, c.width, b->row_bytes,
                              w, obs, b->stream));
    return AV_OK;
}

av_status av_step(av_batch_t b, const uint8_t *actions, float *rewards, uint8_t *done) {
    g_last_error.clear();
    return step_k(b, 1, actions, rewards, done);
}

av_status av_step_n(av_batch_t b, int32_t k, const uint8_t *actions, float *rewards,
                    uint8_t *done) {
    g_last_error.clear();
    return step_k(b, k, actions, rewards, done);
}

av_status av_step_observe(av_batch_t b, int32_t k, const uint8_t *actions, float *rewards,
                          uint8_t *done, int32_t w, uint8_t *obs) {
    g_last_error.clear();
    if (!b) return fail(AV_EINVAL, "batch handle is NULL");
    if (!obs) return fail(AV_EINVAL, "obs is NULL");
    if (w < 1 || w > 255) return fail(AV_EINVAL, "window size %d outside [1, 255]", w);
    return step_k(b, k, actions, rewards, done, obs, w);
}

av_status av_get_maps(av_batch_t b, uint8_t *dst) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    if (!dst) return fail(AV_EINVAL, "dst is NULL");
    if (av_status st = set_device(b)) return st;
    const av_config &c = b->cfg;
    AV_HIP(launch_unpack(b->d_state, dst, c.num_envs, c.channels, c.height, c.width, b->row_bytes,
                         b->stream));
    return AV_OK;
}

av_status av_observe(av_batch_t b, int32_t w, uint8_t *dst) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    if (!dst) return fail(AV_EINVAL, "dst is NULL");
    if (w < 1 || w > 255) return fail(AV_EINVAL, "window size %d outside [1, 255]", w);
    if (!b->have_maps) return fail(AV_ESTATE, "call av_reset first");
    if (av_status st = set_device(b)) return st;
    const av_config &c = b->cfg;
    AV_HIP(launch_observe(b->d_state, c.num_envs, c.channels, c.height, c.width, b->row_bytes, w,
                          dst, b->stream));
    return AV_OK;
}

av_status av_rule_features(av_batch_t b, uint8_t *dst) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    if (!dst) return fail(AV_EINVAL, "dst is NULL");
    if (!b->have_rules) return fail(AV_ESTATE, "call av_load_rules first");
    if (av_status st = set_device(b)) return st;
    if (!b->features.empty())
        AV_HIP(hipMemcpyAsync(dst, b->features.data(), b->features.size(), hipMemcpyHostToDevice,
                              b->stream));
    AV_HIP(hipStreamSynchronize(b->stream));
    return AV_OK;
}

static MutateArgs mutate_args(const av_mutation &m) {
    MutateArgs a;
    a.seed = m.seed; a.generation = m.generation;
    a.map_flip_p32 = m.map_flip_p32; a.map_channels = m.map_channels;
    a.entry_p32 = m.entry_p32; a.entry_channels = m.entry_channels;
    a.reward_p32 = m.reward_p32; a.reward_lo = m.reward_lo; a.reward_hi = m.reward_hi;
    return a;
}

av_status av_mutate_maps(const uint8_t *src, uint8_t *dst, int32_t n, int32_t channels,
                         int32_t height, int32_t width, const av_mutation *m, int32_t device,
                         void *stream) {
    g_last_error.clear();
    if (!m) return fail(AV_EINVAL, "mutation parameters are NULL");
    if (n < 0 || channels < 1 || channels > 31 || height < 1 || height > kMaxDim || width < 1 ||
        width > kMaxDim)
        return fail(AV_EINVAL, "sizes out of range: n %d, C %d, H %d, W %d", n, channels, height,
                    width);
    if (n > 0 && (!src || !dst)) return fail(AV_EINVAL, "src and dst must not be NULL");
    AV_HIP(hipSetDevice(device));
    AV_HIP(launch_mutate_maps(src, dst, n, channels, height, width, mutate_args(*m),
                              static_cast<hipStream_t>(stream)));
    return AV_OK;
}

av_status av_mutate_rules(int32_t num_sets, int32_t num_rules, int32_t channels,
                          int32_t max_pat_h, int32_t max_pat_w, const int32_t *shape,
                          const int8_t *in_src, const int8_t *out_src, const int32_t *reward_src,
                          int8_t *in_dst, int8_t *out_dst, int32_t *reward_dst,
                          const av_mutation *m, int32_t device, void *stream) {
    g_last_error.clear();
    if (!m) return fail(AV_EINVAL, "mutation parameters are NULL");
    if (num_sets < 0 || num_rules < 0 || num_rules > kMaxRules || channels < 1 || channels > 31 ||
        max_pat_h < 1 ||
        max_pat_h > kMaxPat || max_pat_w < 1 || max_pat_w > kMaxPat)
        return fail(AV_EINVAL, "sizes out of range: S %d, R %d, C %d, pattern %d x %d", num_sets,
                    num_rules, channels, max_pat_h, max_pat_w);
    if (m->reward_lo > m->reward_hi)
        return fail(AV_EINVAL, "reward_lo %d > reward_hi %d", m->reward_lo, m->reward_hi);
    if (int64_t(num_sets) * num_rules > 0 &&
        (!shape || !in_src || !out_src || !reward_src || !in_dst || !out_dst || !reward_dst))
        return fail(AV_EINVAL, "rule arrays must not be NULL");
    AV_HIP(hipSetDevice(device));
    AV_HIP(launch_mutate_rules(num_sets, num_rules, channels, max_pat_h, max_pat_w, shape, in_src,
                               out_src, reward_src, in_dst, out_dst, reward_dst, mutate_args(*m),
                               static_cast<hipStream_t>(stream)));
    return AV_OK;
}

const void *av_state_ptr(av_batch_t b) {
    g_last_error.clear();
    if (!b) { fail(AV_EINVAL, "batch handle is NULL"); return nullptr; }
    return b->d_state;
}

av_status av_get_info(av_batch_t b, av_info *info) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    if (!info) return fail(AV_EINVAL, "info is NULL");
    info->num_envs = b->cfg.num_envs;
    info->height = b->cfg.height;
    info->width = b->cfg.width;
    info->channels = b->cfg.channels;
    info->row_bytes = b->row_bytes;
    info->engine = b->engine;
    info->state_bytes = b->state_bytes;
    info->blob_bytes = sizeof(BlobHeader) + 2 * b->state_bytes + sizeof(int32_t) * b->cfg.num_envs;
    return AV_OK;
}

av_status av_get_state(av_batch_t b, void *host_blob, size_t *bytes) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    if (!bytes) return fail(AV_EINVAL, "bytes is NULL");
    const size_t need = sizeof(BlobHeader) + 2 * b->state_bytes + sizeof(int32_t) * b->cfg.num_envs;
    if (!host_blob) { *bytes = need; return AV_OK; }
    if (*bytes < need) return fail(AV_EINVAL, "blob needs %zu bytes, got %zu", need, *bytes);
    if (av_status st = set_device(b)) return st;
    BlobHeader h{};
    std::memcpy(h.magic, kBlobMagic, 8);
    h.B = b->cfg.num_envs; h.H = b->cfg.height; h.W = b->cfg.width; h.C = b->cfg.channels;
    h.row_bytes = b->row_bytes; h.state_bytes = b->state_bytes;
    char *p = static_cast<char *>(host_blob);
    AV_HIP(hipStreamSynchronize(b->stream));
    AV_HIP(hipMemcpy(&h.step_no, b->d_n, sizeof(uint64_t), hipMemcpyDeviceToHost));   // copy 0
    std::memcpy(p, &h, sizeof h);
    AV_HIP(hipMemcpy(p + sizeof h, b->d_state, b->state_bytes, hipMemcpyDeviceToHost));
    AV_HIP(hipMemcpy(p + sizeof h + b->state_bytes, b->d_init, b->state_bytes, hipMemcpyDeviceToHost));
    AV_HIP(hipMemcpy(p + sizeof h + 2 * b->state_bytes, b->d_t, sizeof(int32_t) * b->cfg.num_envs,
                     hipMemcpyDeviceToHost));
    *bytes = need;
    return AV_OK;
}

av_status av_set_state(av_batch_t b, const void *host_blob, size_t bytes) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    if (!host_blob) return fail(AV_EINVAL, "host_blob is NULL");
    const size_t need = sizeof(BlobHeader) + 2 * b->state_bytes + sizeof(int32_t) * b->cfg.num_envs;
    if (bytes < need) return fail(AV_EINVAL, "blob has %zu bytes, need %zu", bytes, need);
    BlobHeader h;
    std::memcpy(&h, host_blob, sizeof h);
    if (std::memcmp(h.magic, kBlobMagic, 8) != 0) return fail(AV_EINVAL, "not a state blob");
    if (h.B != b->cfg.num_envs || h.H != b->cfg.height || h.W != b->cfg.width ||
        h.C != b->cfg.channels || h.row_bytes != b->row_bytes || h.state_bytes != b->state_bytes)
        return fail(AV_EINVAL, "blob is for a %d x %dx%d x %d batch", h.B, h.H, h.W, h.C);
    if (av_status st = set_device(b)) return st;
    const char *p = static_cast<const char *>(host_blob);
    AV_HIP(hipStreamSynchronize(b->stream));
    AV_HIP(hipMemcpy(b->d_state, p + sizeof h, b->state_bytes, hipMemcpyHostToDevice));
    AV_HIP(hipMemcpy(b->d_init, p + sizeof h + b->state_bytes, b->state_bytes, hipMemcpyHostToDevice));
    AV_HIP(hipMemcpy(b->d_t, p + sizeof h + 2 * b->state_bytes, sizeof(int32_t) * b->cfg.num_envs,
                     hipMemcpyHostToDevice));
    AV_HIP(launch_fill_counters(nullptr, 0, b->d_n, step_copies(b->cfg.num_envs), 0, h.step_no,
                                b->stream));
    AV_HIP(hipStreamSynchronize(b->stream));
    b->have_maps = true;
    return AV_OK;
}

av_status av_set_stream(av_batch_t b, void *stream) {
    g_last_error.clear();
    if (av_status st = check_batch(b)) return st;
    b->stream = static_cast<hipStream_t>(stream);
    b->cfg.stream = stream;
    return AV_OK;
}

av_status av_destroy_batch(av_batch_t b) {
    g_last_error.clear();
    if (!b) return AV_OK;
    av_status st = AV_OK;
    if (hipSetDevice(b->cfg.device) == hipSuccess) {
        hipError_t e = hipStreamSynchronize(b->stream);
        if (e != hipSuccess) st = fail(AV_EDEVICE, "hipStreamSynchronize: %s", hipGetErrorString(e));
        free_device_program(b);
        free_control(b);
        dev_free(b->d_state);
        dev_free(b->d_init);
        dev_free(b->d_t);
        dev_free(b->d_n);
        dev_free(b->d_order);
        dev_free(b->d_cost);
        if (b->h_order) (void)hipHostFree(b->h_order);
        if (b->h_cost) (void)hipHostFree(b->h_cost);
        if (b->cost_ev) (void)hipEventDestroy(b->cost_ev);
    }
    delete b;
    return st;
}

}  // extern "C"
