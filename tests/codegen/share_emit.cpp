// Emits bit-sliced "at least K" counts of several term lists through the lane16 generator's
// shared adders (codegen::Gen::share, then at_least per list) as a C++ function, for the CPU
// test of the generator.  Lists are drawn from a seed: each holds a term of its own (the
// channel's old value), terms of a common pool (the shifted match words) as they are (plus
// votes) or complemented (minus votes), and its threshold is the number of complemented terms
// plus one, as in the write; a second kind of list takes random terms and thresholds.
#include <cstdio>
#include <random>
#include <string>
#include <vector>

#include "codegen.h"

int main(int argc, char **argv) {
    const unsigned seed = argc > 1 ? unsigned(std::stoul(argv[1])) : 1u;
    std::mt19937 rng(seed);
    const int pool = 24 + int(rng() % 40), lists = 1 + int(rng() % 7);
    av::codegen::Gen g;
    std::vector<std::vector<av::codegen::Gen::Bit>> terms(lists);
    std::vector<long> K(lists);
    for (int l = 0; l < lists; ++l) {
        const bool write_like = (rng() % 4) != 0;
        long minus = 0;
        if (write_like) terms[l].push_back({"x[" + std::to_string(pool + l) + "]", false});
        for (int t = 0; t < pool; ++t) {
            if (rng() % 10 < 3) continue;             // not voted on this list
            const bool inv = rng() % 2;
            minus += inv;
            terms[l].push_back({"x[" + std::to_string(t) + "]", inv});
        }
        if (terms[l].empty()) terms[l].push_back({"x[0]", false});
        const long n = long(terms[l].size());
        K[l] = write_like ? minus + 1 : 1 + long(rng() % n);
    }
    if (argc > 2 && std::string(argv[2]) == "ops") {
        // adders emitted with and without sharing
        av::codegen::Gen alone;
        for (int l = 0; l < lists; ++l) alone.at_least(terms[l], K[l]);
        std::vector<av::codegen::Gen::Levels> lv = g.share(terms);
        for (int l = 0; l < lists; ++l) g.at_least(lv[l], K[l]);
        auto ops = [](const std::string &t) {
            size_t n = 0;
            for (size_t at = t.find("bitop3"); at != std::string::npos; at = t.find("bitop3", at + 1)) ++n;
            return n;
        };
        std::printf("%zu %zu\n", ops(g.o.str()), ops(alone.o.str()));
        return 0;
    }
    std::vector<av::codegen::Gen::Levels> lv = g.share(terms);
    for (int l = 0; l < lists; ++l) {
        g.o << "{\n";
        g.at_least(lv[l], K[l]);
        g.o << "out[" << l << "] = GT;\n}\n";
    }
    std::printf("#define NIN %d\n#define NOUT %d\n", pool + lists, lists);
    std::printf("static const int kTerms[NOUT][%d] = {", pool + lists + 1);
    // per list: its terms as (index + 1) * (complemented ? -1 : 1), 0-terminated
    for (int l = 0; l < lists; ++l) {
        std::printf("%s{", l ? ", " : "");
        for (const auto &b : terms[l]) {
            const int idx = std::stoi(b.name.substr(2, b.name.size() - 3));
            std::printf("%d, ", b.inv ? -(idx + 1) : idx + 1);
        }
        std::printf("0}");
    }
    std::printf("};\nstatic const long kK[NOUT] = {");
    for (int l = 0; l < lists; ++l) std::printf("%s%ld", l ? ", " : "", K[l]);
    std::printf("};\nstatic void counts(const u32 *x, u32 *out) {\n%s}\n", g.o.str().c_str());
    return 0;
}
