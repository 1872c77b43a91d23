// Executor rewrites: the plan's phases become executed phases, with copies
// folded into the steps that produce their data where that saves traffic or
// launches.  Host only.
#include <algorithm>
#include <map>
#include <tuple>
#include <vector>

#include "exec_state.hpp"

namespace arp {

// What the reads and writes of one executed phase touch, kept up to date
// while copies of later phases are folded into its reduce steps (each fold
// adds writes only): per buffer, the touched intervals by begin, with the
// step that touches them and whether it writes them.  Folding phase after
// phase then costs the added writes only.
struct Merged {
    struct Touch { int64_t end; size_t step; bool write; };
    std::vector<std::multimap<int64_t, Touch>> iv;  // per buffer
    std::vector<int64_t> maxlen;                    // longest interval per buffer
    std::vector<bool> reduce;                       // per step: two or more sources
    std::vector<int32_t> extra;                     // per step: destinations one fold adds

    Merged(const XPhase& ph, int32_t n)
        : iv(size_t(n)), maxlen(size_t(n), 0), extra(ph.steps.size(), 0) {
        for (size_t i = 0; i < ph.steps.size(); ++i) {
            const XStep& st = ph.steps[i];
            reduce.push_back(st.srcs.size() >= 2);
            if (st.end <= st.begin) continue;
            for (int32_t q : st.srcs) touch(q, st.begin, st.end, i, false);
            for (int32_t d : st.dsts) touch(d, st.begin, st.end, i, true);
        }
    }
    void touch(int32_t buf, int64_t b, int64_t e, size_t step, bool write) {
        iv[size_t(buf)].insert({b, Touch{e, step, write}});
        maxlen[size_t(buf)] = std::max(maxlen[size_t(buf)], e - b);
    }
    // the reduce step that writes `buf` from position b on (its end in
    // `end`), or -1
    int64_t producer(int32_t buf, int64_t b, int64_t& end) const {
        const auto r = iv[size_t(buf)].equal_range(b);
        for (auto it = r.first; it != r.second; ++it)
            if (it->second.write && reduce[it->second.step]) {
                end = it->second.end;
                return int64_t(it->second.step);
            }
        return -1;
    }
    // does `step` already write `buf` (from its begin b on)?
    bool writes(int32_t buf, int64_t b, size_t step) const {
        const auto r = iv[size_t(buf)].equal_range(b);
        for (auto it = r.first; it != r.second; ++it)
            if (it->second.write && it->second.step == step) return true;
        return false;
    }
    // does a step other than `self` touch positions [b, e) of `buf`?
    bool other(int32_t buf, int64_t b, int64_t e, size_t self) const {
        if (e <= b) return false;
        const auto& m = iv[size_t(buf)];
        for (auto it = m.lower_bound(b - maxlen[size_t(buf)]); it != m.end() && it->first < e; ++it)
            if (it->second.end > b && it->second.step != self) return true;
        return false;
    }
};

// Executed phases of a plan.  With `fuse`, two rewrites remove memory
// traffic or launches without changing any result (subject to kFuseDst /
// kFuseBytes of exec_state.hpp):
//  * multicast: copies in one phase that read the same range of the same
//    buffer become one step that reads it once and stores it to every
//    destination;
//  * reduce-then-broadcast: when every step of phase q+1 copies a range that
//    is a union of ranges the reduce steps of phase q have just produced,
//    the copies are absorbed into those reduce steps, which then store their
//    results to the copies' destinations as well, and phase q+1 disappears
//    (the last ReduceScatter phase and the first AllGather phase meet this
//    way).  Applied again with q+2, q+3, ... as long as it succeeds, so that
//    a whole AllGather can fold into the last reduce phase (RHD: each eighth
//    is reduced once and stored to all eight buffers).  The absorbed writes
//    are checked against every read and write of the other steps of phase q,
//    so the merged phase stays free of hazards.
std::vector<XPhase> exec_phases(const Plan& p, bool fuse) {
    std::vector<XPhase> ph(size_t(p.num_phases()));
    for (int32_t q = 0; q < p.num_phases(); ++q) {
        ph[size_t(q)].plan_phase = q;
        for (int64_t i = p.phase_first[size_t(q)]; i < p.phase_first[size_t(q) + 1]; ++i) {
            const Step& st = p.steps[size_t(i)];
            XStep x;
            x.begin = st.begin;
            x.end = st.end;
            x.srcs.assign(p.srcs.begin() + st.src_off, p.srcs.begin() + st.src_off + st.nsrc);
            x.dsts = {st.dst};
            ph[size_t(q)].steps.push_back(std::move(x));
        }
    }
    if (!fuse) return ph;
    auto copy_bytes = [&](const XPhase& xp) {
        int64_t b = 0;
        for (const XStep& x : xp.steps)
            if (x.srcs.size() == 1) b += 2 * int64_t(x.dsts.size()) * (x.end - x.begin) * p.esize;
        return b;
    };
    for (XPhase& xp : ph) {  // multicast
        const bool small = copy_bytes(xp) <= kFuseBytes;
        std::map<std::tuple<int32_t, int64_t, int64_t>, size_t> first;
        std::vector<XStep> kept;
        for (XStep& x : xp.steps) {
            if (x.srcs.size() == 1 && x.end > x.begin) {
                auto key = std::make_tuple(x.srcs[0], x.begin, x.end);
                auto it = first.find(key);
                if (it != first.end()) {
                    XStep& m = kept[it->second];
                    m.dsts.insert(m.dsts.end(), x.dsts.begin(), x.dsts.end());
                    continue;
                }
                first.emplace(key, kept.size());
            }
            kept.push_back(std::move(x));
        }
        if (!small) {  // undo groups that grew past kFuseDst destinations
            std::vector<XStep> undone;
            for (XStep& x : kept) {
                if (x.srcs.size() == 1 && int32_t(x.dsts.size()) > kFuseDst) {
                    for (int32_t d : x.dsts) {
                        XStep y;
                        y.begin = x.begin;
                        y.end = x.end;
                        y.srcs = x.srcs;
                        y.dsts = {d};
                        undone.push_back(std::move(y));
                    }
                } else {
                    undone.push_back(std::move(x));
                }
            }
            kept = std::move(undone);
        }
        xp.steps = std::move(kept);
    }
    // reduce-then-broadcast, transitively: phase q absorbs q+1, then q+2, ...
    // as long as each next phase consists of copies whose source ranges are
    // exactly unions of ranges the (merged) reduce steps of q write
    auto absorb = [&](XPhase& cur, Merged& m, const XPhase& nxt) {
        // copies whose reads are all distinct move data nobody reads twice:
        // folding them into the reduce steps saves their reads entirely
        const bool small = copy_bytes(nxt) <= kFuseBytes;
        bool distinct = true;
        {
            std::vector<std::tuple<int32_t, int64_t, int64_t>> rd;
            for (const XStep& c : nxt.steps) {
                if (c.end <= c.begin) continue;
                if (c.dsts.size() != 1) distinct = false;
                for (int32_t q : c.srcs) rd.emplace_back(q, c.begin, c.end);
            }
            std::sort(rd.begin(), rd.end());
            for (size_t i = 1; i < rd.size() && distinct; ++i)
                if (std::get<0>(rd[i]) == std::get<0>(rd[i - 1]) &&
                    std::get<1>(rd[i]) < std::get<2>(rd[i - 1]))
                    distinct = false;
        }
        // (producer step, destination) pairs to add, checked against the
        // merged phase as it stands before this fold
        std::vector<std::pair<size_t, int32_t>> adds;
        struct Reset {  // leaves m.extra all zero on every return
            Merged& m;
            const std::vector<std::pair<size_t, int32_t>>& adds;
            ~Reset() { for (const auto& ad : adds) m.extra[ad.first] = 0; }
        } reset{m, adds};
        bool any = false;
        for (const XStep& c : nxt.steps) {
            if (c.end <= c.begin) continue;  // empty step: nothing to move
            if (c.srcs.size() != 1) return false;
            any = true;
            int64_t at = c.begin;
            while (at < c.end) {
                int64_t end = 0;
                const int64_t i = m.producer(c.srcs[0], at, end);
                if (i < 0 || end > c.end) return false;
                for (int32_t d : c.dsts) {
                    if (m.other(d, at, end, size_t(i))) return false;
                    adds.emplace_back(size_t(i), d);
                    m.extra[size_t(i)] += 1;
                }
                at = end;
            }
        }
        if (!any) return false;
        if (!small && !distinct)
            for (const auto& ad : adds)
                if (int32_t(cur.steps[ad.first].dsts.size()) + m.extra[ad.first] > kFuseDst)
                    return false;
        for (const auto& ad : adds) {
            XStep& s = cur.steps[ad.first];
            if (!m.writes(ad.second, s.begin, ad.first)) {
                s.dsts.push_back(ad.second);
                m.touch(ad.second, s.begin, s.end, ad.first, true);
            }
        }
        return true;
    };
    for (size_t q = 0; q + 1 < ph.size(); ++q) {
        if (ph[q].steps.empty()) continue;
        bool copies = false;  // only a phase of copies can be folded
        for (const XStep& c : ph[q + 1].steps) {
            if (c.srcs.size() != 1 && c.end > c.begin) {
                copies = false;
                break;
            }
            copies = copies || c.end > c.begin;
        }
        if (!copies) continue;
        Merged m(ph[q], p.n);
        for (size_t j = q + 1; j < ph.size(); ++j) {
            if (!absorb(ph[q], m, ph[j])) break;
            ph[j].steps.clear();
        }
    }
    std::vector<XPhase> out;
    for (XPhase& xp : ph)
        if (!xp.steps.empty()) out.push_back(std::move(xp));
    return out;
}

// Is every executed phase free of hazards?  A step may read and write the
// same positions (each lane loads all sources before storing); otherwise no
// step may touch what another step of its phase writes.
bool exec_phases_hazard_free(const std::vector<XPhase>& ph, int32_t n, std::string& why) {
    for (size_t q = 0; q < ph.size(); ++q) {
        const Touches all(ph[q], n, true, true);
        for (size_t i = 0; i < ph[q].steps.size(); ++i) {
            const XStep& st = ph[q].steps[i];
            for (int32_t d : st.dsts)
                if (all.other(d, st.begin, st.end, i)) {
                    why = "executed phase " + std::to_string(q) + ": step " + std::to_string(i) +
                          " writes what another step touches";
                    return false;
                }
        }
    }
    return true;
}

}  // namespace arp
