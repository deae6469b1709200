// The lane16 engine: maps of at most 16 x 16, one map row per lane, two maps per 32-bit
// lane word.  Declarations shared by the host library and the engine.
#pragma once

#include <cstdint>
#include <vector>

#include "av_internal.h"

namespace av {

constexpr int kLane16MaxPat = 4;

struct Lane16Rule {
    int n = 1, m = 1, reward = 0;
    std::vector<int8_t> in, out;   // [C+1][n][m], tri-valued
};

struct Lane16Program {
    bool ready = false;
};

struct Lane16Device {
    void *unused = nullptr;
};

inline bool lane16_eligible(const av_config &) { return false; }
inline void lane16_compile(const std::vector<std::vector<Lane16Rule>> &, int, Lane16Program &p) {
    p.ready = false;
}
inline hipError_t lane16_upload(const Lane16Program &, Lane16Device &) { return hipSuccess; }
inline void lane16_free(Lane16Device &) {}
inline hipError_t launch_lane16_step(const StepArgs &, const Lane16Device &, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace av
