// Pieces of the rule-set-to-kernel-code generator (lane16): pattern entries in rarest-first
// order, the vote of one pattern cell, how many entries a rule is probed with, and the
// emitter of bit-sliced vote counts.
#pragma once

#include <algorithm>
#include <cstdlib>
#include <deque>
#include <map>
#include <sstream>
#include <string>
#include <tuple>
#include <vector>

#include "av_internal.h"

namespace av {
namespace codegen {

// One specified input entry of a rule: channel c (C = the force plane) at pattern row i,
// column j must be `want`; `rank` orders entries rarest first.
struct Entry {
    int c, i, j, want, rank;
};

// Rarest evidence first: force and player bits are rare, walls and empty tiles common;
// a must-be-1 entry rejects more anchors than a must-be-0 entry.
inline int rank_of(int c, int want, int C) {
    int ch;
    if (c == C) ch = 0;
    else if (c == kChPlayer) ch = 1;
    else if (c == kChGoal || c >= 4) ch = 2;
    else if (c == kChWall) ch = 3;
    else ch = 4;
    return (want ? 0 : 8) + ch;
}

// The vote K_O of one pattern cell-channel: +1, -1 or 0 (in, out in {-1 = don't care, 0, 1}).
inline int kout(int in, int out) {
    if (out < 0) return 0;
    if (out == 1) return in == 1 ? 0 : 1;
    return in == 0 ? 0 : -1;
}

// A vote of rule r at pattern row i, column j.
struct Vote {
    int r, i, j;
};

// Number of entries a loaded rule is probed with before the wave-wide test: at least two, at
// most four, more while a static guess of the share of waves (`maps` maps each) in which
// some anchor passes them stays above 10 %.  The guess uses the synthetic maps' statistics:
// one player cell per map with its force cell beside it, walls on 30 % of the cells, the
// other tile types sharing the rest evenly.  It only decides how much of a rule runs before
// the test, never what the rule computes.
inline size_t probe_len(const std::vector<Entry> &es, int C, int H, int W, int n, int m, int maps) {
    const double cells = double(H) * W, anchors = double(H - n + 1) * (W - m + 1);
    const size_t lo = std::min<size_t>(2, es.size()), hi = std::min<size_t>(4, es.size());
    size_t k = 0;
    double p = anchors;
    for (; k < hi; ++k) {
        if (k >= lo && maps * p <= 0.1) break;
        const Entry &en = es[k];
        double q1;
        if (en.c == C || en.c == kChPlayer) {
            q1 = 1.0 / cells;
            for (size_t f = 0; f < k; ++f) {            // a force cell beside a player cell
                const Entry &o = es[f];
                const bool pair = (en.c == C && o.c == kChPlayer) || (en.c == kChPlayer && o.c == C);
                if (pair && o.want && en.want && std::abs(o.i - en.i) + std::abs(o.j - en.j) == 1)
                    q1 = 0.25;
            }
        } else if (en.c == kChWall) {
            q1 = 0.3;
        } else {
            q1 = 0.7 / std::max(1, C - 2);
        }
        p *= en.want ? q1 : 1.0 - q1;
    }
    return k;
}

// Emits straight-line code into `o`; `type` is the lane word type of the generated kernel.
class Gen {
  public:
    std::ostringstream o;
    std::string type = "u32";
    int tmp = 0;
    std::string fresh() { return "t" + std::to_string(tmp++); }

    // Bit-sliced population count of `terms` (each a plane word): returns the count's bits,
    // least significant first, built from full and half adders.
    std::vector<std::string> count(const std::vector<std::string> &terms) {
        std::vector<std::deque<std::string>> lv(1, std::deque<std::string>(terms.begin(), terms.end()));
        std::vector<std::string> bits;
        for (size_t k = 0; k < lv.size(); ++k) {
            std::deque<std::string> q = lv[k];
            std::vector<std::string> carries;
            while (q.size() >= 3) {
                const std::string a = q[0], b = q[1], c = q[2];
                q.pop_front(); q.pop_front(); q.pop_front();
                const std::string s = fresh(), cy = fresh();
                o << "const " << type << " " << s << " = " << a << " ^ " << b << " ^ " << c << ";\n";
                o << "const " << type << " " << cy << " = (" << a << " & " << b << ") | (" << c
                  << " & (" << a << " ^ " << b << "));\n";
                q.push_back(s);
                carries.push_back(cy);
            }
            if (q.size() == 2) {
                const std::string a = q[0], b = q[1];
                const std::string s = fresh(), cy = fresh();
                o << "const " << type << " " << s << " = " << a << " ^ " << b << ";\n";
                o << "const " << type << " " << cy << " = " << a << " & " << b << ";\n";
                q.clear();
                q.push_back(s);
                carries.push_back(cy);
            }
            bits.push_back(q.empty() ? std::string("0") : q.front());
            if (!carries.empty()) {
                if (lv.size() == k + 1) lv.emplace_back();
                lv[k + 1].insert(lv[k + 1].end(), carries.begin(), carries.end());
            }
        }
        return bits;
    }

    // One term of a bit-sliced sum: a plane word, possibly complemented.
    struct Bit {
        std::string name;
        bool inv = false;
        std::string expr() const { return inv ? "(~" + name + ")" : name; }
    };

    // v_bitop3 truth table of f over three operands, each possibly complemented: bit
    // (4 a + 2 b + c) of the table is f(a, b, c) for operand bits a, b, c (the first operand
    // is the table index's high bit).
    template <typename F>
    static int table3(F f, bool i0, bool i1, bool i2) {
        int t = 0;
        for (int k = 0; k < 8; ++k) {
            const int a = ((k >> 2) & 1) ^ int(i0), b = ((k >> 1) & 1) ^ int(i1), c = (k & 1) ^ int(i2);
            t |= (f(a, b, c) & 1) << k;
        }
        return t;
    }

    // A bit-sliced sum in progress: level k holds terms of weight 2^k.
    using Levels = std::vector<std::deque<Bit>>;

    static int sum3(int a, int b, int c) { return a ^ b ^ c; }
    static int maj3(int a, int b, int c) { return (a & b) | (a & c) | (b & c); }
    Bit op3(const Bit &a, const Bit &b, const Bit &c, int table) {
        const std::string r = fresh();
        o << "const " << type << " " << r << " = __builtin_amdgcn_bitop3_b32(" << a.name << ", "
          << b.name << ", " << c.name << ", 0x" << std::hex << table << std::dec << ");\n";
        return Bit{r, false};
    }

    // Carry-save sums of several term lists started together: a full adder over three terms
    // that several lists hold serves them all.  Its inputs may be complemented in one list and
    // not in another as long as all three are (the sum and carry of complements are the
    // complements of the sum and carry), so a list takes the adder's outputs complemented
    // then.  Greedy, level by level: the signed pairs held by the most lists, each widened to
    // the third term most of their holders share, until no three terms are held by two lists;
    // a shared sum stays on its level (it may be shared again), a shared carry moves up one.
    // Only terms that several lists hold are added here; the rest is left to at_least.
    std::vector<Levels> share(const std::vector<std::vector<Bit>> &lists) {
        std::vector<Levels> lv(lists.size());
        for (size_t l = 0; l < lists.size(); ++l)
            lv[l].emplace_back(lists[l].begin(), lists[l].end());
        auto find = [](const std::deque<Bit> &q, const std::string &n) {
            for (size_t x = 0; x < q.size(); ++x)
                if (q[x].name == n) return int(x);
            return -1;
        };
        for (size_t k = 0;; ++k) {
            bool any_level = false;
            for (auto &L : lv) any_level |= L.size() > k;
            if (!any_level) break;
            for (;;) {
                // signed pairs (names in order, relative complement) and the lists holding them
                std::map<std::tuple<std::string, std::string, bool>, std::vector<int>> pairs;
                for (size_t l = 0; l < lv.size(); ++l) {
                    if (lv[l].size() <= k) continue;
                    const std::deque<Bit> &q = lv[l][k];
                    for (size_t x = 0; x < q.size(); ++x)
                        for (size_t y = x + 1; y < q.size(); ++y) {
                            const Bit &a = q[x].name < q[y].name ? q[x] : q[y];
                            const Bit &b = q[x].name < q[y].name ? q[y] : q[x];
                            pairs[{a.name, b.name, a.inv != b.inv}].push_back(int(l));
                        }
                }
                std::vector<std::pair<size_t, std::tuple<std::string, std::string, bool>>> order;
                for (auto &pr : pairs)
                    if (pr.second.size() >= 2) order.push_back({pr.second.size(), pr.first});
                if (order.empty()) break;
                std::stable_sort(order.begin(), order.end(),
                                 [](const auto &u, const auto &v) { return u.first > v.first; });
                // the best triple among the most held pairs: (holders, a, b, c, c relative to a)
                size_t best_n = 0;
                std::string ba, bb, bc;
                bool bab = false, bac = false;
                for (size_t t = 0; t < order.size() && t < 8; ++t) {
                    const auto &[na, nb, ab] = order[t].second;
                    std::map<std::pair<std::string, bool>, size_t> third;
                    for (int l : pairs[order[t].second]) {
                        const std::deque<Bit> &q = lv[l][k];
                        const bool ia = q[find(q, na)].inv;
                        for (const Bit &c : q)
                            if (c.name != na && c.name != nb) ++third[{c.name, c.inv != ia}];
                    }
                    for (auto &tc : third)
                        if (tc.second > best_n) {
                            best_n = tc.second;
                            ba = na; bb = nb; bab = ab;
                            bc = tc.first.first; bac = tc.first.second;
                        }
                }
                if (best_n < 2) break;
                // one adder, inputs as the first holder has them
                Bit s{}, cy{};
                bool first = true, first_ia = false;
                for (size_t l = 0; l < lv.size(); ++l) {
                    if (lv[l].size() <= k) continue;
                    std::deque<Bit> &q = lv[l][k];
                    const int xa = find(q, ba), xb = find(q, bb), xc = find(q, bc);
                    if (xa < 0 || xb < 0 || xc < 0) continue;
                    const Bit a = q[xa], b = q[xb], c = q[xc];
                    if ((a.inv != b.inv) != bab || (a.inv != c.inv) != bac) continue;
                    if (first) {
                        s = op3(a, b, c, table3(sum3, a.inv, b.inv, c.inv));
                        cy = op3(a, b, c, table3(maj3, a.inv, b.inv, c.inv));
                        first_ia = a.inv;
                        first = false;
                    }
                    const bool flip = a.inv != first_ia;
                    std::deque<Bit> rest;
                    for (size_t x = 0; x < q.size(); ++x)
                        if (int(x) != xa && int(x) != xb && int(x) != xc) rest.push_back(q[x]);
                    rest.push_back(Bit{s.name, flip});
                    q = rest;
                    if (lv[l].size() == k + 1) lv[l].emplace_back();
                    lv[l][k + 1].push_back(Bit{cy.name, flip});
                }
            }
        }
        return lv;
    }

    // The cells where the number of set terms is at least K (K >= 1): the terms are added
    // with a carry-save tree of full adders (sum and carry are one v_bitop3 each, with the
    // terms' complements folded into the truth tables) and the count's bits are compared with
    // the constant K; emitted as GT.
    void at_least(const std::vector<Bit> &terms, long K) {
        at_least(Levels(1, std::deque<Bit>(terms.begin(), terms.end())), K);
    }
    // The same for a sum already started (share): terms of weight 2^k on level k.
    void at_least(Levels lv, long K) {
        std::vector<Bit> bits;
        auto xor2 = [](int a, int b, int) { return a ^ b; };
        auto and2 = [](int a, int b, int) { return a & b; };
        for (size_t k = 0; k < lv.size(); ++k) {
            std::deque<Bit> q = lv[k];
            std::vector<Bit> carries;
            while (q.size() >= 3) {
                const Bit a = q[0], b = q[1], c = q[2];
                q.pop_front(); q.pop_front(); q.pop_front();
                q.push_back(op3(a, b, c, table3(sum3, a.inv, b.inv, c.inv)));
                carries.push_back(op3(a, b, c, table3(maj3, a.inv, b.inv, c.inv)));
            }
            if (q.size() == 2) {
                const Bit a = q[0], b = q[1];
                q.clear();
                q.push_back(op3(a, b, a, table3(xor2, a.inv, b.inv, a.inv)));
                carries.push_back(op3(a, b, a, table3(and2, a.inv, b.inv, a.inv)));
            }
            bits.push_back(q.empty() ? Bit{"0u", false} : q.front());
            if (!carries.empty()) {
                if (lv.size() == k + 1) lv.emplace_back();
                lv[k + 1].insert(lv[k + 1].end(), carries.begin(), carries.end());
            }
        }
        const size_t m = bits.size();
        if (m < 63 && K >= (1L << m)) {
            o << type << " GT = 0u;\n";
            return;
        }
        // count >= K: from the high bit down, EQ holds where the count's bits so far equal K's,
        // GE where they already exceed them
        o << type << " GT = 0u, EQ = ~(" << type << ")0u;\n";
        for (size_t k = m; k-- > 0;) {
            if ((K >> k) & 1) o << "EQ &= " << bits[k].expr() << ";\n";
            else o << "GT |= EQ & " << bits[k].expr() << ";\n";
        }
        o << "GT |= EQ;\n";
    }

    // The cells where old + #plus > #minus: a bit-sliced comparison of two counts (bits least
    // significant first), emitted as GT; the caller declares nothing.
    void greater(const std::vector<std::string> &P, const std::vector<std::string> &N) {
        const size_t K = std::max(P.size(), N.size());
        o << type << " GT = 0, EQ = ~(" << type << ")0;\n";
        for (size_t k = K; k-- > 0;) {
            const std::string pk = k < P.size() ? P[k] : "0", nk = k < N.size() ? N[k] : "0";
            o << "GT |= EQ & " << pk << " & ~" << nk << ";\n";
            o << "EQ &= ~(" << pk << " ^ " << nk << ");\n";
        }
    }
};

}  // namespace codegen
}  // namespace av
