// lane16 engine, host side: turns a shared rule set into the straight-line body of the
// step kernel, compiles the kernel with hipRTC for gfx950 and launches it.
//
// Generated code, per rule r (n x m), all on 32-bit lane words that hold one map row of
// two environments (see lane16_kernel.hip):
//   M_r  = valid-anchor mask V_n_m (rows y <= H-n, columns x <= W-m of both halves),
//          AND-ed with every specified input entry (c, i, j, want): plane c moved up i rows
//          (DPP row shift) and right-aligned by j columns, complemented for want = 0.  This
//          is the paper's thresholded convolution (Sec. 2.1) evaluated 32 anchors at a time.
//          The two rarest entries are tested first; if no anchor of the wave survives them
//          the rest of the rule is skipped (a wave-uniform branch).
//   reward += reward_r * popcount(M_r) per half.
//   votes: every nonzero K_O = O - I entry (c, i, j) moves M_r down i rows and left by j
//          columns onto the cells it writes; +1 votes are OR-ed into PL_c, -1 votes into
//          MI_c.  A cell with votes of one sign only takes that sign's value; if some cell
//          of the wave has votes of both signs, the channel's votes are counted exactly with
//          carry-save adders and the cell becomes 1 iff old + sum >= 1 (Sec. 2.1
//          transposed-convolution write, clamped to {0, 1}), counted as old + #plus +
//          #(minus terms that are 0) >= #minus + 1; full adders over terms that several
//          channels count are formed once for all of them.
//   The force plane's own votes are not evaluated: the plane is dropped after the step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <map>
#include <set>
#include <sstream>
#include <string>
#include <vector>

#include "codegen.h"
#include "jit.h"
#include "lane16.h"

namespace av {
namespace {

using codegen::Entry;
using codegen::Gen;
using codegen::Vote;
using codegen::kout;
using codegen::rank_of;

#include "_lane16_template.inc"   // kLane16Template: lane16_kernel.hip as a string

std::string plane(int c, int C) { return c == C ? std::string("F") : "p[" + std::to_string(c) + "]"; }

// Rule application control for rule r on its match word `M` (paper Sec. 2.1.1), after its
// matches are complete and before its reward and votes.  `applied(q)` names the final match
// word of an earlier rule q.
//   inhibition: anchors of r whose n x m patch overlaps the patch of an applied match of q:
//     rows y - nq + 1 .. y + n - 1 of q OR-ed (DPP row shifts), then dilated over columns
//     x - mq + 1 .. x + m - 1 inside each 16-bit half, and cleared from M;
//   cap K: per half, an inclusive prefix sum of the lanes' popcounts across the 16-lane row
//     (Hillis-Steele with DPP row shifts; two 16-bit counters in one word); a lane whose
//     prefix exceeds K keeps only the lowest K - (exclusive prefix) bits of its half, so the
//     first K matches in row-major order survive.
template <typename Applied>
void emit_control(std::ostringstream &o, int r, const std::string &M,
                  const std::vector<Lane16Rule> &rules, const Lane16Control &ctl,
                  Applied applied) {
    const Lane16Rule &ru = rules[r];
    for (int q : ctl.inhibitors[r]) {
        const Lane16Rule &rq = rules[q];
        o << "{ // rule " << q << " inhibits rule " << r << "\n";
        o << "u32 O = " << applied(q) << ";\n";
        for (int d = 1; d < ru.n; ++d) o << "O |= DPP_SHL(" << applied(q) << ", " << d << ");\n";
        for (int d = 1; d < rq.n; ++d) o << "O |= DPP_SHR(" << applied(q) << ", " << d << ");\n";
        o << "u32 D = O;\n";
        for (int k = 1; k < ru.m; ++k) o << "D |= (O >> " << k << ") & BOTH(0xFFFFu >> " << k << ");\n";
        for (int k = 1; k < rq.m; ++k)
            o << "D |= (O << " << k << ") & BOTH((0xFFFFu << " << k << ") & 0xFFFFu);\n";
        o << M << " &= ~D;\n}\n";
    }
    const int K = ctl.limit[r];
    if (K > 0 && ctl.random) {
        // random site order: K rounds of a row-wide maximum over the random keys of the
        // remaining matches of each environment whose match count exceeds K
        o << "{ // rule " << r << ": at most " << K << " matches, largest random index first\n";
        o << "const u32 cnt = (u32)__popc(" << M << " & 0xFFFFu) | ((u32)__popc(" << M << " >> 16) << 16);\n";
        o << "u32 tot = cnt;\ntot += (u32)DPP_ROR((int)tot, 1);\ntot += (u32)DPP_ROR((int)tot, 2);\n"
             "tot += (u32)DPP_ROR((int)tot, 4);\ntot += (u32)DPP_ROR((int)tot, 8);\n";
        o << "const bool exA = (tot & 0xFFFFu) > " << K << "u, exB = (tot >> 16) > " << K << "u;\n";
        o << "if (ANY(u32(exA || exB))) {\n";
        o << "if (!keys_ready) { site_keys(kb, y, eA, eB, hasA, hasB, nstep, seed); keys_ready = true; }\n";
        o << "u32 remA = exA ? (" << M << " & 0xFFFFu) : 0u, remB = exB ? (" << M << " >> 16) : 0u;\n";
        o << "u32 keep = (exA ? 0u : (" << M << " & 0xFFFFu)) | (exB ? 0u : (" << M << " & 0xFFFF0000u));\n";
        o << "for (int t = 0; t < " << K << "; ++t) {\n"
             "u32 bA = 0u, bB = 0u;\n"
             "for (u32 x = remA; x; x &= x - 1u) bA = max(bA, kb[__ffs(x) - 1]);\n"
             "for (u32 x = remB; x; x &= x - 1u) bB = max(bB, kb[16 + __ffs(x) - 1]);\n"
             "u32 mA = bA, mB = bB;\n";
        for (int d : {1, 2, 4, 8})
            o << "mA = max(mA, (u32)DPP_ROR((int)mA, " << d << ")); mB = max(mB, (u32)DPP_ROR((int)mB, "
              << d << "));\n";
        o << "if (bA != 0u && bA == mA)\n"
             "for (u32 x = remA; x; x &= x - 1u) { const u32 b = x & (0u - x); "
             "if (kb[__ffs(x) - 1] == mA) { remA ^= b; keep |= b; break; } }\n";
        o << "if (bB != 0u && bB == mB)\n"
             "for (u32 x = remB; x; x &= x - 1u) { const u32 b = x & (0u - x); "
             "if (kb[16 + __ffs(x) - 1] == mB) { remB ^= b; keep |= b << 16; break; } }\n";
        o << "}\n" << M << " = keep;\n}\n}\n";
    } else if (K > 0) {
        o << "{ // rule " << r << ": at most " << K << " matches, first in row-major order\n";
        o << "const u32 cnt = (u32)__popc(" << M << " & 0xFFFFu) | ((u32)__popc(" << M << " >> 16) << 16);\n";
        o << "u32 inc = cnt;\ninc += DPP_SHR(inc, 1);\ninc += DPP_SHR(inc, 2);\n"
             "inc += DPP_SHR(inc, 4);\ninc += DPP_SHR(inc, 8);\n";
        o << "const int incA = int(inc & 0xFFFFu), incB = int(inc >> 16);\n";
        o << "if (ANY(u32((incA > " << K << ") | (incB > " << K << ")))) {\n";
        o << "int kA = " << K << " - (incA - int(cnt & 0xFFFFu)), kB = " << K
          << " - (incB - int(cnt >> 16));\n";
        o << "u32 xa = " << M << " & 0xFFFFu, xb = " << M << " >> 16, keep = 0u;\n";
        o << "for (int t = 0; t < 16; ++t) {\n"
             "const u32 ba = xa & (0u - xa), bb = xb & (0u - xb);\n"
             "if (kA > 0 && ba) { keep |= ba; --kA; }\n"
             "if (kB > 0 && bb) { keep |= bb << 16; --kB; }\n"
             "xa ^= ba; xb ^= bb;\n}\n";
        o << M << " = keep;\n}\n}\n";
    }
}

bool controlled(const Lane16Control *ctl, int r) {
    return ctl && (ctl->limit[r] > 0 || !ctl->inhibitors[r].empty());
}

}  // namespace

bool lane16_eligible(const av_config &c) {
    return c.height <= 16 && c.width <= 16 && c.per_env_rules == 0 && c.max_pat_h <= 16 &&
           c.max_pat_w <= 16;
}

std::string lane16_rules_body(int C, int H, int W, const std::vector<Lane16Rule> &rules,
                              const Lane16Control *ctl) {
    Gen g;
    std::ostringstream &o = g.o;
    const int C1 = C + 1, R = int(rules.size());
    auto in_at = [&](const Lane16Rule &r, int c, int i, int j) {
        return int(r.in[(size_t(c) * r.n + i) * r.m + j]);
    };
    auto out_at = [&](const Lane16Rule &r, int c, int i, int j) {
        return int(r.out[(size_t(c) * r.n + i) * r.m + j]);
    };

    std::vector<std::vector<Entry>> ents(R);
    std::set<std::pair<int, int>> xs, shapes;
    std::vector<std::vector<Vote>> plus(C), minus(C);
    std::vector<std::vector<std::pair<Vote, int>>> rule_votes(R);   // (vote, channel * 2 + sign)
    for (int r = 0; r < R; ++r) {
        const Lane16Rule &ru = rules[r];
        shapes.insert({ru.n, ru.m});
        for (int c = 0; c < C1; ++c)
            for (int i = 0; i < ru.n; ++i)
                for (int j = 0; j < ru.m; ++j) {
                    const int w = in_at(ru, c, i, j);
                    if (w >= 0) {
                        ents[r].push_back({c, i, j, w, rank_of(c, w, C)});
                    }
                    const int k = c < C ? kout(w, out_at(ru, c, i, j)) : 0;
                    if (k > 0) plus[c].push_back({r, i, j});
                    if (k < 0) minus[c].push_back({r, i, j});
                    if (k) rule_votes[r].push_back({Vote{r, i, j}, c * 2 + (k > 0)});
                }
        std::stable_sort(ents[r].begin(), ents[r].end(),
                         [](const Entry &a, const Entry &b) { return a.rank < b.rank; });
    }
    // Column-shifted planes read on every step (by the moves and by the loaded rules' probe
    // entries) are computed once up front; the others only inside the branches that need them.
    const int n_fixed = std::min(R, kMoveRules);
    std::vector<size_t> probe(R);
    for (int r = 0; r < R; ++r) {
        probe[r] = r < n_fixed ? ents[r].size()
                               : codegen::probe_len(ents[r], C, H, W, rules[r].n, rules[r].m, 8);
        for (size_t e = 0; e < probe[r]; ++e)
            if (ents[r][e].j > 0) xs.insert({ents[r][e].c, ents[r][e].j});
    }

    o << "// ---- generated: " << R << " rules over " << C1 << " planes ----\n";
    for (auto &x : xs)
        o << "const u32 X" << x.first << "_" << x.second << " = " << plane(x.first, C) << " >> "
          << x.second << ";\n";
    for (auto &s : shapes)
        o << "const u32 V" << s.first << "_" << s.second << " = (y <= " << (H - s.first)
          << ") ? BOTH(COLMASK(" << std::max(0, W - s.second + 1) << ")) : 0u;\n";

    auto base = [&](const Entry &e) {
        if (!e.j) return plane(e.c, C);
        if (xs.count({e.c, e.j})) return "X" + std::to_string(e.c) + "_" + std::to_string(e.j);
        return "(" + plane(e.c, C) + " >> " + std::to_string(e.j) + ")";
    };

    auto row_and = [&](const std::vector<Entry> &es) {
        std::string q;
        for (const Entry &en : es) {
            if (!q.empty()) q += " & ";
            q += (en.want ? "" : "~") + base(en);
        }
        return q;
    };
    auto emit_rows = [&](const std::string &M, const std::vector<Entry> &es) {
        std::map<int, std::vector<Entry>> by_row;
        for (const Entry &en : es) by_row[en.i].push_back(en);
        for (auto &row : by_row) {
            if (row.first == 0) o << M << " &= " << row_and(row.second) << ";\n";
            else o << M << " &= DPP_SHL(" << row_and(row.second) << ", " << row.first << ");\n";
        }
    };
    // a loaded rule that casts votes marks the step (wave-uniform: set only under ballots)
    const bool track = R > n_fixed;
    auto emit_votes = [&](int r) {
        const std::string M = "M" + std::to_string(r);
        std::set<int> js;
        for (auto &v : rule_votes[r])
            if (v.first.j) js.insert(v.first.j);
        for (int j : js) o << "const u32 L" << r << "_" << j << " = " << M << " << " << j << ";\n";
        for (auto &v : rule_votes[r]) {
            const int c = v.second / 2;
            const bool pl = v.second & 1;
            const std::string src = v.first.j ? "L" + std::to_string(r) + "_" + std::to_string(v.first.j) : M;
            const std::string t = v.first.i ? "DPP_SHR(" + src + ", " + std::to_string(v.first.i) + ")" : src;
            o << (pl ? "PL" : "MI") << c << " |= " << t << ";\n";
        }
        if (r >= n_fixed && !rule_votes[r].empty()) o << "lf = true;\n";
    };
    auto emit_reward = [&](int r) {
        const std::string M = "M" + std::to_string(r);
        if (rules[r].reward != 0)
            o << "rA += " << rules[r].reward << " * (int)__popc(" << M << " & 0xFFFFu); rB += "
              << rules[r].reward << " * (int)__popc(" << M << " >> 16); paid = true;\n";
    };

    // The built-in moves (rules 0..3) are cheap and fire in most waves: evaluated in full,
    // without branches.  Loaded rules are probed with their rarest entries; one wave-uniform
    // test over all probes skips the rest when no anchor survives anywhere.
    for (int r = 0; r < R; ++r) {
        const Lane16Rule &ru = rules[r];
        const std::string M = "M" + std::to_string(r);
        o << "u32 " << M << " = V" << ru.n << "_" << ru.m << ";\n";
        if (r < n_fixed) {
            emit_rows(M, ents[r]);
            continue;
        }
        for (size_t e = 0; e < probe[r]; ++e) {
            const Entry &en = ents[r][e];
            const std::string t = en.i ? "DPP_SHL(" + base(en) + ", " + std::to_string(en.i) + ")" : base(en);
            o << M << " &= " << (en.want ? "" : "~") << t << ";\n";
        }
    }
    // The moves' vote words live for the whole step; those of channels only loaded rules vote
    // on exist inside the probe test's branch only.
    std::vector<std::vector<Vote>> mpl(C), mmi(C);
    for (int c = 0; c < C; ++c) {
        for (const Vote &v : plus[c])
            if (v.r < n_fixed) mpl[c].push_back(v);
        for (const Vote &v : minus[c])
            if (v.r < n_fixed) mmi[c].push_back(v);
    }
    auto moves_vote = [&](int c) { return !mpl[c].empty() || !mmi[c].empty(); };
    auto any_vote = [&](int c) { return !plus[c].empty() || !minus[c].empty(); };
    for (int c = 0; c < C; ++c)
        if (track ? moves_vote(c) : any_vote(c))
            o << "u32 PL" << c << " = 0u, MI" << c << " = 0u;\n";
    for (int r = 0; r < n_fixed; ++r) {
        emit_reward(r);
        emit_votes(r);
    }
    if (track) {
        o << "bool lf = false;\n";
        o << "if (ANY(";
        for (int r = n_fixed; r < R; ++r) o << (r > n_fixed ? " | " : "") << "M" << r;
        o << ")) {\n";
        for (int c = 0; c < C; ++c)
            if (any_vote(c) && !moves_vote(c)) o << "u32 PL" << c << " = 0u, MI" << c << " = 0u;\n";
        for (int r = n_fixed; r < R; ++r) {
            const std::string M = "M" + std::to_string(r);
            const size_t pr = probe[r];
            if (controlled(ctl, r)) {
                // complete the matches, filter them, then pay and vote with what is left
                if (ents[r].size() > pr) {
                    o << "if (ANY(" << M << ")) {\n";
                    emit_rows(M, std::vector<Entry>(ents[r].begin() + pr, ents[r].end()));
                    o << "}\n";
                }
                o << "if (ANY(" << M << ")) {\n";
                emit_control(o, r, M, rules, *ctl,
                             [](int q) { return "M" + std::to_string(q); });
                o << "if (ANY(" << M << ")) {\n";
                emit_reward(r);
                emit_votes(r);
                o << "}\n}\n";
                continue;
            }
            o << "if (ANY(" << M << ")) {\n";
            if (ents[r].size() > pr) {
                emit_rows(M, std::vector<Entry>(ents[r].begin() + pr, ents[r].end()));
                o << "if (ANY(" << M << ")) {\n";
            }
            emit_reward(r);
            emit_votes(r);
            if (ents[r].size() > pr) o << "}\n";
            o << "}\n";
        }
    }

    // The write.  A cell with votes of one sign only takes that sign's value; if some cell of
    // the wave got votes of both signs on a channel, the channel's votes are counted exactly.
    // `pl` / `mi` list the votes that can be nonzero on the path being emitted.
    auto emit_write = [&](const std::vector<std::vector<Vote>> &pl,
                          const std::vector<std::vector<Vote>> &mi) {
        std::vector<int> voted, both;
        for (int c = 0; c < C; ++c) {
            if (pl[c].empty() && mi[c].empty()) continue;
            voted.push_back(c);
            if (!pl[c].empty() && !mi[c].empty()) both.push_back(c);
        }
        // the one-sign result of every plane comes first, off the exact-count branch's path
        for (int c : voted)
            o << "u32 N" << c << " = (p[" << c << "] | PL" << c << ") & ~MI" << c << ";\n";
        auto tname = [](int r, int i, int j) {
            return "T" + std::to_string(r) + "_" + std::to_string(i) + "_" + std::to_string(j);
        };
        if (!both.empty()) {
            // Exact counts, in waves where some cell of some channel got votes of both signs.
            // Every match word moved onto the cells it votes on is formed once for all the
            // channels; then each mixed channel becomes old + #plus - #minus >= 1, counted as
            // old + #plus + #(minus terms that are 0) >= #minus + 1 (one carry-save count).
            o << "if (ANY(";
            for (size_t k = 0; k < both.size(); ++k)
                o << (k ? " | " : "") << "(PL" << both[k] << " & MI" << both[k] << ")";
            o << ")) {\n";
            std::set<std::pair<int, int>> shifts;
            std::set<std::tuple<int, int, int>> terms;
            for (int c : both)
                for (auto *lst : {&pl[c], &mi[c]})
                    for (const Vote &v : *lst) {
                        if (v.j) shifts.insert({v.r, v.j});
                        terms.insert({v.r, v.i, v.j});
                    }
            for (auto &sh : shifts)
                o << "const u32 E" << sh.first << "_" << sh.second << " = M" << sh.first << " << "
                  << sh.second << ";\n";
            for (auto &t : terms) {
                const int r = std::get<0>(t), i = std::get<1>(t), j = std::get<2>(t);
                const std::string src = j ? "E" + std::to_string(r) + "_" + std::to_string(j) : "M" + std::to_string(r);
                o << "const u32 " << tname(r, i, j) << " = "
                  << (i ? "DPP_SHR(" + src + ", " + std::to_string(i) + ")" : src) << ";\n";
            }
            // the channels' counts start together: full adders over terms that several
            // channels share (a shifted match word votes on about five channels of a dense
            // rule set) are formed once; each mixed channel finishes its own count
            std::vector<std::vector<Gen::Bit>> lists;
            for (int c : both) {
                std::vector<Gen::Bit> cnt{{"p[" + std::to_string(c) + "]", false}};
                for (const Vote &v : pl[c]) cnt.push_back({tname(v.r, v.i, v.j), false});
                for (const Vote &v : mi[c]) cnt.push_back({tname(v.r, v.i, v.j), true});
                lists.push_back(std::move(cnt));
            }
            std::vector<Gen::Levels> started = g.share(lists);
            for (size_t k = 0; k < both.size(); ++k) {
                const int c = both[k];
                o << "if (ANY(PL" << c << " & MI" << c << ")) { // channel " << c << ": "
                  << pl[c].size() << " + votes, " << mi[c].size() << " - votes\n";
                g.at_least(started[k], long(mi[c].size()) + 1);
                o << "N" << c << " = GT;\n}\n";
            }
            o << "}\n";
        }
        for (int c : voted) o << "p[" << c << "] = N" << c << ";\n";
    };
    if (track) {
        // Steps where a loaded rule voted write inside the probe test's branch; all others
        // (most steps of sparse rule sets) write only the moves' channels and count only the
        // moves' votes.
        o << "if (lf) {\n";
        emit_write(plus, minus);
        o << "}\n}\nif (!lf) {\n";
        emit_write(mpl, mmi);
        o << "}\n";
    } else {
        emit_write(plus, minus);
    }
    o << "(void)F;\n";
    return o.str();
}

// Sequential rule order: one block per rule, in list order.  Each block derives its shifted
// planes from the map as the rules before it left it (force plane included), matches the
// rule, and applies its votes (exactly counted where its own matches overlap with both
// signs) before the next block.
std::string lane16_rules_body_sequential(int C, int H, int W, const std::vector<Lane16Rule> &rules,
                                         const Lane16Control *ctl = nullptr) {
    Gen g;
    std::ostringstream &o = g.o;
    const int C1 = C + 1, R = int(rules.size());
    auto in_at = [&](const Lane16Rule &r, int c, int i, int j) {
        return int(r.in[(size_t(c) * r.n + i) * r.m + j]);
    };
    auto out_at = [&](const Lane16Rule &r, int c, int i, int j) {
        return int(r.out[(size_t(c) * r.n + i) * r.m + j]);
    };
    std::set<std::pair<int, int>> shapes;
    for (const Lane16Rule &ru : rules) shapes.insert({ru.n, ru.m});
    o << "// ---- generated: " << R << " rules in sequence over " << C1 << " planes ----\n";
    for (auto &s : shapes)
        o << "const u32 V" << s.first << "_" << s.second << " = (y <= " << (H - s.first)
          << ") ? BOTH(COLMASK(" << std::max(0, W - s.second + 1) << ")) : 0u;\n";

    // final match words of the rules that inhibit later ones
    std::vector<bool> inhibits(R, false);
    if (ctl)
        for (int r = 0; r < R; ++r)
            for (int q : ctl->inhibitors[r]) inhibits[q] = true;
    for (int r = 0; r < R; ++r)
        if (inhibits[r]) o << "u32 A" << r << " = 0u;\n";

    for (int r = 0; r < R; ++r) {
        const Lane16Rule &ru = rules[r];
        std::vector<Entry> ents;
        std::set<std::pair<int, int>> xs;
        std::vector<std::vector<Vote>> plus(C1), minus(C1);
        for (int c = 0; c < C1; ++c)
            for (int i = 0; i < ru.n; ++i)
                for (int j = 0; j < ru.m; ++j) {
                    const int w = in_at(ru, c, i, j);
                    if (w >= 0) {
                        ents.push_back({c, i, j, w, rank_of(c, w, C)});
                        if (j > 0) xs.insert({c, j});
                    }
                    const int k = kout(w, out_at(ru, c, i, j));
                    if (k > 0) plus[c].push_back({r, i, j});
                    if (k < 0) minus[c].push_back({r, i, j});
                }
        std::stable_sort(ents.begin(), ents.end(),
                         [](const Entry &a, const Entry &b) { return a.rank < b.rank; });
        auto base = [&](const Entry &e) {
            return e.j ? "X" + std::to_string(e.c) + "_" + std::to_string(e.j) : plane(e.c, C);
        };
        auto row_and = [&](const std::vector<Entry> &es) {
            std::string q;
            for (const Entry &en : es) {
                if (!q.empty()) q += " & ";
                q += (en.want ? "" : "~") + base(en);
            }
            return q;
        };
        auto emit_rows = [&](const std::vector<Entry> &es) {
            std::map<int, std::vector<Entry>> by_row;
            for (const Entry &en : es) by_row[en.i].push_back(en);
            for (auto &row : by_row) {
                if (row.first == 0) o << "M &= " << row_and(row.second) << ";\n";
                else o << "M &= DPP_SHL(" << row_and(row.second) << ", " << row.first << ");\n";
            }
        };
        bool writes = false;
        for (int c = 0; c < C1; ++c) writes |= !plus[c].empty() || !minus[c].empty();
        if (!writes && ru.reward == 0 && !inhibits[r]) continue;   // no effect at all

        o << "{ // rule " << r << "\n";
        for (auto &x : xs)
            o << "const u32 X" << x.first << "_" << x.second << " = " << plane(x.first, C) << " >> "
              << x.second << ";\n";
        o << "u32 M = V" << ru.n << "_" << ru.m << ";\n";
        const bool fixed = r < kMoveRules;
        const size_t probe = fixed ? ents.size() : std::min<size_t>(2, ents.size());
        int open = 0;
        if (fixed) {
            emit_rows(ents);
        } else {
            for (size_t e = 0; e < probe; ++e) {
                const Entry &en = ents[e];
                const std::string t = en.i ? "DPP_SHL(" + base(en) + ", " + std::to_string(en.i) + ")" : base(en);
                o << "M &= " << (en.want ? "" : "~") << t << ";\n";
            }
            o << "if (ANY(M)) {\n";
            ++open;
            if (ents.size() > probe) {
                emit_rows(std::vector<Entry>(ents.begin() + probe, ents.end()));
                o << "if (ANY(M)) {\n";
                ++open;
            }
        }
        if (controlled(ctl, r))
            emit_control(o, r, "M", rules, *ctl, [](int q) { return "A" + std::to_string(q); });
        if (inhibits[r]) o << "A" << r << " = M;\n";
        if (ru.reward != 0)
            o << "rA += " << ru.reward << " * (int)__popc(M & 0xFFFFu); rB += " << ru.reward
              << " * (int)__popc(M >> 16); paid = true;\n";
        // votes of this rule
        std::set<int> js;
        std::vector<int> touched, both;
        for (int c = 0; c < C1; ++c) {
            if (plus[c].empty() && minus[c].empty()) continue;
            touched.push_back(c);
            if (!plus[c].empty() && !minus[c].empty()) both.push_back(c);
            for (auto *lst : {&plus[c], &minus[c]})
                for (const Vote &v : *lst)
                    if (v.j) js.insert(v.j);
        }
        for (int j : js) o << "const u32 L" << j << " = M << " << j << ";\n";
        auto term = [&](const Vote &v) {
            const std::string src = v.j ? "L" + std::to_string(v.j) : std::string("M");
            return v.i ? "DPP_SHR(" + src + ", " + std::to_string(v.i) + ")" : src;
        };
        for (int c : touched) {
            o << "u32 PL" << c << " = 0u, MI" << c << " = 0u;\n";
            for (const Vote &v : plus[c]) o << "PL" << c << " |= " << term(v) << ";\n";
            for (const Vote &v : minus[c]) o << "MI" << c << " |= " << term(v) << ";\n";
            o << "u32 N" << c << " = (" << plane(c, C) << " | PL" << c << ") & ~MI" << c << ";\n";
        }
        if (!both.empty()) {
            o << "u32 CF = 0u;\n";
            for (int c : both) o << "CF |= PL" << c << " & MI" << c << ";\n";
            o << "if (ANY(CF)) {\n";
            std::set<std::pair<int, int>> tset;
            for (int c : both)
                for (auto *lst : {&plus[c], &minus[c]})
                    for (const Vote &v : *lst) tset.insert({v.i, v.j});
            auto tname = [](int i, int j) { return "T" + std::to_string(i) + "_" + std::to_string(j); };
            for (auto &t : tset)
                o << "const u32 " << tname(t.first, t.second) << " = " << term(Vote{r, t.first, t.second})
                  << ";\n";
            for (int c : both) {
                // old + #plus - #minus >= 1, counted as old + #plus + #(minus terms that are
                // 0) >= #minus + 1
                std::vector<Gen::Bit> cnt{{plane(c, C), false}};
                for (const Vote &v : plus[c]) cnt.push_back({tname(v.i, v.j), false});
                for (const Vote &v : minus[c]) cnt.push_back({tname(v.i, v.j), true});
                o << "{ // plane " << c << "\n";
                g.at_least(cnt, long(minus[c].size()) + 1);
                o << "N" << c << " = GT;\n}\n";
            }
            o << "}\n";
        }
        for (int c : touched) o << plane(c, C) << " = N" << c << ";\n";
        for (; open > 0; --open) o << "}\n";
        o << "}\n";
    }
    return o.str();
}

void lane16_compile(const std::vector<std::vector<Lane16Rule>> &sets, int C, int H, int W, int L,
                    bool sequential, Lane16Program &p, const Lane16Control *ctl) {
    std::string src = kLane16Template;
    std::ostringstream d;
    d << "#define AV_C " << C << "\n#define AV_H " << H << "\n#define AV_W " << W << "\n#define AV_L "
      << L << "\n";
    bool pays = false;
    for (const Lane16Rule &r : sets.at(0)) pays |= r.reward != 0;
    if (!pays) d << "#define AV_NO_REWARD 1\n";
    auto put = [&](const std::string &marker, const std::string &text) {
        const size_t at = src.find(marker);
        if (at != std::string::npos) src.replace(at, marker.size(), text);
    };
    bool random = false;
    if (ctl && ctl->random)
        for (size_t r = 0; r < ctl->limit.size(); ++r) random |= ctl->limit[r] > 0;
    put("/*@DEFINES@*/", d.str());
    put("/*@PHILOX@*/", random ? std::string("#define AV_RANDOM_SITES 1\n") + kPhiloxSource : std::string());
    put("/*@RULES@*/", sequential ? lane16_rules_body_sequential(C, H, W, sets.at(0), ctl)
                                  : lane16_rules_body(C, H, W, sets.at(0), ctl));
    p.source = std::move(src);
}

hipError_t lane16_upload(const Lane16Program &p, Lane16Device &d, std::string *log) {
    return jit_kernel(p.source, "av_lane16.hip", "av_lane16_step", &d.fn, log);
}

hipError_t launch_lane16_step(const StepArgs &a, const Lane16Device &d, hipStream_t s) {
    if (!d.fn) return hipErrorInvalidDeviceFunction;
    const int waves = (a.B + 7) / 8;               // eight environments per wave
    const unsigned blocks = unsigned((waves + 3) / 4);
    void *state = a.state;
    const void *init = a.init;
    int *t = a.t;
    const uint8_t *actions = a.actions;
    float *rewards = a.rewards;
    uint8_t *done = a.done;
    int B = a.B, K = a.k;
    unsigned long long seed = a.ctl.seed;
    uint64_t *nctr = a.nctr;
    uint8_t *obs = a.obs;
    int w = a.obs_w;
    const void *gsrc = a.gsrc;
    int gnf = a.gnf, gA = a.gA;
    const int32_t *gdepth = a.gdepth;
    void *args[] = {&state, &init, &t, &actions, &rewards, &done, &B, &K, &seed, &nctr,
                    &obs, &w, &gsrc, &gnf, &gA, &gdepth};
    // dynamic LDS: the fused observation's window buffers, four waves of eight environments
    const unsigned lds = obs ? unsigned(4 * ((8 * a.C * w * w + 16 + 15) & ~15)) : 0u;
    return hipModuleLaunchKernel(d.fn, blocks, 1, 1, 256, 1, 1, lds, s, args, nullptr);
}

}  // namespace av
