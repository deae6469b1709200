// av_step_n_static (include/autoverse.h): k steps of caller-owned environments that allocate
// no device memory, for callers that cannot allocate.
//
// The work is av_step_n's on the wave or generic engine.  What av_create_batch and
// av_load_rules would allocate and the kernels read besides the caller's inputs and outputs
// (the compiled rule program, and the launch units' copies of the batch step number, which
// the kernels store but read only for rule application control, which this entry point does
// not offer) lives in one file-scope device array, `scratch`, of kScratchBytes.  Its device
// address is taken once per device with hipGetSymbolAddress (the array's name in host code is
// only a host-side stand-in) and passed to the kernels like any other buffer.
//
// Every call on a device shares that device's array: calls that overlap on one device (on
// different streams, or from several threads) race on it.  The rule program is copied into
// it on the call's stream (from pageable host memory, so the copy waits for the stream's
// earlier work, which may still read the previous program, and the host image is free when
// the call returns).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "av_internal.h"

using namespace av;

namespace {

constexpr size_t kScratchBytes = size_t(4) << 20;   // AV_STATIC_SCRATCH_BYTES
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];   // device address of `scratch` on each device, once taken

av_status scratch_on(int device, void **out) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) {
            char m[160];
            std::snprintf(m, sizeof m, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
            return set_error(AV_EDEVICE, m);
        }
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return AV_OK;
}

size_t round256(size_t n) { return (n + 255) & ~size_t(255); }

}  // namespace

extern "C" av_status av_step_n_static(const av_config *cfg, int32_t num_rules,
                                      const int32_t *shape, const int8_t *in_pat,
                                      const int8_t *out_pat, const int32_t *reward, void *state,
                                      const void *init, int32_t *counters, int32_t k,
                                      const uint8_t *actions, float *rewards, uint8_t *done) {
    set_error(AV_OK, "");
    if (!cfg) return set_error(AV_EINVAL, "cfg is NULL");
    const av_config &c = *cfg;
    char m[256];
    if (c.num_envs < 1 || c.height < 1 || c.height > kMaxDim || c.width < 1 ||
        c.width > kMaxDim || c.channels < 4 || c.channels > 31 || c.max_pat_h < 1 ||
        c.max_pat_h > kMaxPat || c.max_pat_w < 1 || c.max_pat_w > kMaxPat ||
        c.max_episode_steps < 0 || (c.per_env_rules != 0 && c.per_env_rules != 1)) {
        std::snprintf(m, sizeof m, "sizes out of range: B %d, %d x %d, C %d, patterns %d x %d, "
                      "L %d, per_env_rules %d", c.num_envs, c.height, c.width, c.channels,
                      c.max_pat_h, c.max_pat_w, c.max_episode_steps, c.per_env_rules);
        return set_error(AV_EINVAL, m);
    }
    if (c.rule_mode != AV_RULES_PARALLEL && c.rule_mode != AV_RULES_SEQUENTIAL)
        return set_error(AV_EINVAL, "unknown rule_mode");
    if (c.engine != AV_ENGINE_AUTO && c.engine != AV_ENGINE_WAVE && c.engine != AV_ENGINE_GENERIC)
        return set_error(AV_EINVAL, "av_step_n_static runs the wave or the generic engine only");
    if (num_rules < 0 || num_rules > c.max_rules || c.max_rules > kMaxRules)
        return set_error(AV_EINVAL, "num_rules outside [0, max_rules] or max_rules above 252");
    if (num_rules > 0 && (!shape || !in_pat || !out_pat || !reward))
        return set_error(AV_EINVAL, "rule arrays must not be NULL");
    if (k < 1) return set_error(AV_EINVAL, "k must be >= 1");
    if (!state || !init || !counters || !actions || !rewards || !done)
        return set_error(AV_EINVAL, "state, init, counters, actions, rewards and done must not be "
                         "NULL");
    const int Rt = num_rules + kMoveRules;
    const size_t env_lds = generic_env_lds_bytes(c.height, c.width, c.channels, Rt);
    if (env_lds > size_t(kLdsBudget))
        return set_error(AV_EINVAL, "one environment's working set exceeds 64 KiB of LDS");
    const bool wave_fits =
        wave_lds_bytes(c.height, c.width, c.channels, Rt) <= size_t(kLdsBudget);
    if (c.engine == AV_ENGINE_WAVE && !wave_fits)
        return set_error(AV_EINVAL, "the wave engine's LDS working set exceeds 64 KiB");
    if (c.device < 0 || c.device >= kMaxDevices) return set_error(AV_EINVAL, "device out of range");

    std::vector<std::vector<HostRule>> sets;
    if (av_status st = parse_rule_sets(c, num_rules, shape, in_pat, out_pat, reward, sets))
        return st;
    GenericProgram prog;
    compile_generic(sets, c.channels, c.rule_mode == AV_RULES_SEQUENTIAL, prog);

    // scratch image: [step numbers: B + 8 x u64][hdr][votes][match][vote][rvote], each part
    // starting on a 256-byte boundary
    const size_t o_n = 0;
    const size_t o_hdr = round256(o_n + sizeof(uint64_t) * (size_t(c.num_envs) + 8));
    const size_t o_votes = round256(o_hdr + prog.hdr.size() * sizeof(RuleHdr));
    const size_t o_match = round256(o_votes + prog.votes.size() * sizeof(VoteList));
    const size_t o_vote = round256(o_match + prog.match.size() * sizeof(uint32_t));
    const size_t o_rvote = round256(o_vote + prog.vote.size() * sizeof(uint32_t));
    const size_t end = o_rvote + prog.rvote.size() * sizeof(uint32_t);
    if (end > kScratchBytes) {
        std::snprintf(m, sizeof m, "needs %zu bytes of static scratch (8 per environment and the "
                      "compiled rules); the limit is %zu", end, kScratchBytes);
        return set_error(AV_EINVAL, m);
    }
    std::vector<unsigned char> img(end - o_hdr, 0);
    auto put = [&](size_t off, const void *src, size_t n) {
        if (n) std::memcpy(img.data() + (off - o_hdr), src, n);
    };
    put(o_hdr, prog.hdr.data(), prog.hdr.size() * sizeof(RuleHdr));
    put(o_votes, prog.votes.data(), prog.votes.size() * sizeof(VoteList));
    put(o_match, prog.match.data(), prog.match.size() * sizeof(uint32_t));
    put(o_vote, prog.vote.data(), prog.vote.size() * sizeof(uint32_t));
    put(o_rvote, prog.rvote.data(), prog.rvote.size() * sizeof(uint32_t));

    hipError_t e = hipSetDevice(c.device);
    if (e != hipSuccess) return set_error(AV_EDEVICE, hipGetErrorString(e));
    void *base = nullptr;
    if (av_status st = scratch_on(c.device, &base)) return st;
    char *p = static_cast<char *>(base);
    hipStream_t stream = static_cast<hipStream_t>(c.stream);
    e = hipMemcpyAsync(p + o_hdr, img.data(), img.size(), hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return set_error(AV_EDEVICE, hipGetErrorString(e));

    StepArgs a{};
    a.B = c.num_envs; a.H = c.height; a.W = c.width; a.C = c.channels;
    a.L = c.max_episode_steps; a.per_env = c.per_env_rules; a.k = k;
    a.sequential = c.rule_mode == AV_RULES_SEQUENTIAL;
    a.row_bytes = c.width <= 16 ? 2 : (c.width <= 32 ? 4 : 8); a.max_pat_h = c.max_pat_h;
    a.max_pat_w = c.max_pat_w;
    a.state = state; a.init = init; a.t = counters;
    a.nctr = reinterpret_cast<uint64_t *>(p + o_n);
    a.actions = actions; a.rewards = rewards; a.done = done;
    a.prog.hdr = reinterpret_cast<RuleHdr *>(p + o_hdr);
    a.prog.votes = reinterpret_cast<VoteList *>(p + o_votes);
    a.prog.match = reinterpret_cast<uint32_t *>(p + o_match);
    a.prog.vote = reinterpret_cast<uint32_t *>(p + o_vote);
    a.prog.rvote = reinterpret_cast<uint32_t *>(p + o_rvote);
    a.prog.rules_per_set = prog.rules_per_set;
    a.prog.match_stride = prog.match_stride;
    a.prog.vote_stride = prog.vote_stride;
    a.prog.rvote_stride = prog.rvote_stride;
    a.prog.any_reward = prog.any_reward;
    const bool wave = c.engine == AV_ENGINE_WAVE || (c.engine == AV_ENGINE_AUTO && wave_fits);
    if (wave) {
        e = launch_wave_step(a, stream);
    } else {
        const int G = std::max(1, std::min(256 / c.height, int(kLdsBudget / env_lds)));
        e = launch_generic_step(a, G, stream);
    }
    if (e != hipSuccess) return set_error(AV_EDEVICE, hipGetErrorString(e));
    return AV_OK;
}
