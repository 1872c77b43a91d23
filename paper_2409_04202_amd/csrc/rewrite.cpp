// Executor rewrites: the plan's phases become executed phases, with copies
// folded into the steps that produce their data where that saves traffic or
// launches.  Host only.
#include <algorithm>
#include <map>
#include <tuple>
#include <vector>

#include "exec_state.hpp"

namespace arp {

// Executed phases of a plan.  With `fuse`, two rewrites remove memory
// traffic or launches without changing any result (subject to kFuseDst /
// kFuseBytes above):
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
    auto absorb = [&](XPhase& cur, const XPhase& nxt) {
        const Touches touched(cur, p.n, true, true);
        // per buffer, the ranges the reduce steps of cur write, by begin
        std::map<std::pair<int32_t, int64_t>, std::pair<int64_t, size_t>> produced;
        for (size_t i = 0; i < cur.steps.size(); ++i) {
            const XStep& st = cur.steps[i];
            if (st.srcs.size() >= 2 && st.end > st.begin)
                for (int32_t d : st.dsts) produced[{d, st.begin}] = {st.end, i};
        }
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
        // (producer step, destination) pairs to add
        std::vector<std::pair<size_t, int32_t>> adds;
        std::vector<size_t> extra(cur.steps.size(), 0);
        bool any = false;
        for (const XStep& c : nxt.steps) {
            if (c.end <= c.begin) continue;  // empty step: nothing to move
            if (c.srcs.size() != 1) return false;
            any = true;
            int64_t at = c.begin;
            while (at < c.end) {
                auto it = produced.find({c.srcs[0], at});
                if (it == produced.end() || it->second.first > c.end) return false;
                const size_t i = it->second.second;
                for (int32_t d : c.dsts) {
                    if (touched.other(d, at, it->second.first, i)) return false;
                    adds.emplace_back(i, d);
                    extra[i] += 1;
                }
                at = it->second.first;
            }
        }
        if (!any) return false;
        if (!small && !distinct)
            for (size_t i = 0; i < cur.steps.size(); ++i)
                if (int32_t(cur.steps[i].dsts.size() + extra[i]) > kFuseDst) return false;
        for (const auto& ad : adds) {
            XStep& s = cur.steps[ad.first];
            if (std::find(s.dsts.begin(), s.dsts.end(), ad.second) == s.dsts.end())
                s.dsts.push_back(ad.second);
        }
        return true;
    };
    for (size_t q = 0; q + 1 < ph.size(); ++q) {
        if (ph[q].steps.empty()) continue;
        for (size_t j = q + 1; j < ph.size(); ++j) {
            if (!absorb(ph[q], ph[j])) break;
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
