// The lane16 engine: maps of at most 16 x 16 and one rule set shared by every
// environment.  One map row per lane, two maps per 32-bit lane word; the rule set is
// compiled into the kernel at av_load_rules (lane16_kernel.hip is the fixed part).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "av_internal.h"

namespace av {

// One rule in tri-valued form over C + 1 channels: 1 must be / becomes 1, 0 must be /
// becomes 0, -1 don't care.
struct Lane16Rule {
    int n = 1, m = 1, reward = 0;
    std::vector<int8_t> in, out;   // [C+1][n][m]
};

// Rule application control compiled into the lane16 body:
// per rule of the list (moves included, never controlled), a cap on applied matches (0 = all)
// and the earlier rules that inhibit it.
struct Lane16Control {
    std::vector<int> limit;
    std::vector<std::vector<int>> inhibitors;
    bool random = false;           // keep the matches with the largest random index
};

struct Lane16Program {
    std::string source;            // the complete kernel source for this rule set
};

struct Lane16Device {
    hipFunction_t fn = nullptr;    // owned by the process-wide module cache
};

// Maps of at most 16 x 16 (two per lane word, rows within one 16-lane DPP row) and one
// shared rule set (the rules become code).  Pattern extents up to 16 fit DPP row shifts.
bool lane16_eligible(const av_config &c);

// Generate the kernel source for C stored channels, an H x W map, episode length L, the
// rule order (parallel or sequential) and a rule list (the four moves first, then the
// loaded rules).
void lane16_compile(const std::vector<std::vector<Lane16Rule>> &sets, int C, int H, int W,
                    int L, bool sequential, Lane16Program &p,
                    const Lane16Control *ctl = nullptr);

// Compile (hipRTC, gfx950) and load the program on the current device, reusing an
// identical earlier build.  On failure returns an error and the compiler log in *log.
hipError_t lane16_upload(const Lane16Program &p, Lane16Device &d, std::string *log);

inline void lane16_free(Lane16Device &d) { d.fn = nullptr; }

hipError_t launch_lane16_step(const StepArgs &a, const Lane16Device &d, hipStream_t s);

// The generated straight-line rule code alone (exposed for tests of the generator).
std::string lane16_rules_body(int C, int H, int W, const std::vector<Lane16Rule> &rules,
                              const Lane16Control *ctl = nullptr);

}  // namespace av
