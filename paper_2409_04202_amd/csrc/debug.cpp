// Test hooks of the library (csrc/ar_debug.h), host only: a check of the
// executed phases, the launch tiling and the sliced and resident tables
// against the steps, and read-back of the executed steps and of the
// resident programs.
#include <algorithm>
#include <cstring>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "ar_debug.h"
#include "exec_state.hpp"
#include "internal.hpp"

using namespace arp;

// Symbolic check of a streamed slice (stream_kernel): per segment, running
// its program on terms (an input row, an unordered 2-operand add, the
// rounding at the end of a fold) with the buffers' rows in memory and the
// slots in LDS, and with the wave's loads and stores in flight until a wait
// covers them (loads finish in issue order, stores in any order: a wait for
// m finishes every load but the last m issued, and the stores only when m is
// 0), gives every
// buffer the term the executed steps give it phase by phase; no slot is read,
// or written by a fold, while a load into it may be in flight, no row is
// loaded while a store to it may be in flight or stored while a load of it
// may be, no slot beyond the launch's slots is used and no record crosses a
// 64-word chunk.  Per unit: its tile and its segment's program.  Returns ""
// or the first problem.
static std::string check_streamed(const ar_plan& plan, const ExecState& ex, const SliceDesc& sd) {
    const int64_t VEC = 16 / plan.esize;
    const size_t n = size_t(plan.n);
    if (sd.res_waves != 4 || sd.slots < 1 || sd.slots > kStreamMaxSlots || plan.n > kStreamMaxN ||
        int64_t(sd.slots) * 1024 + int64_t(plan.n) * 8 + int64_t(sd.max_nw) * 4 > kLdsBytesPerCU / 2)
        return "streamed launch shape";
    if (int64_t(sd.runits.size()) != sd.nunits || int64_t(sd.tiles.size()) != sd.nunits ||
        int64_t(sd.rec_off.size()) != sd.nseg)
        return "streamed table sizes";
    std::vector<int32_t> words(size_t(sd.nseg), -1);
    for (int64_t i = 0; i < sd.nunits; ++i) {
        const size_t sg = size_t(sd.tiles[size_t(i)].x);
        if (words[sg] < 0) words[sg] = sd.runits[size_t(i)].nw;
    }
    for (int32_t sg = 0; sg < sd.nseg; ++sg) {
        std::map<std::tuple<int, int64_t, int64_t>, int64_t> terms;
        auto term = [&](int kind, int64_t x, int64_t y) {
            if (kind == 1 && x > y) std::swap(x, y);
            return terms.emplace(std::make_tuple(kind, x, y), int64_t(terms.size())).first->second;
        };
        auto fold = [&](const std::vector<int64_t>& v) {
            if (v.size() == 1) return v[0];
            int64_t t = v[0];
            for (size_t j = 1; j < v.size(); ++j) t = term(1, t, v[j]);
            return term(2, t, 0);
        };
        std::vector<int64_t> want(n), hbm(n);
        for (size_t b = 0; b < n; ++b) want[b] = hbm[b] = term(0, int64_t(b), 0);
        bool covered = false;
        for (int32_t q = 0; q < sd.nphases; ++q) {
            std::vector<std::pair<int32_t, int64_t>> outs;
            for (const XStep& x : ex.phases[size_t(sd.p0 + q)].steps) {
                if (!(x.end > x.begin && x.begin <= sd.cuts[size_t(sg)] &&
                      sd.cuts[size_t(sg) + 1] <= x.end))
                    continue;
                covered = true;
                std::vector<int64_t> v;
                for (int32_t b : x.srcs) v.push_back(want[size_t(b)]);
                const int64_t t = fold(v);
                for (int32_t b : x.dsts) outs.push_back({b, t});
            }
            for (const auto& o : outs) want[size_t(o.first)] = o.second;
        }
        const int32_t off = sd.rec_off[size_t(sg)];
        if (!covered) {
            if (off != -1 || words[size_t(sg)] >= 0) return "streamed program on an idle segment";
            continue;
        }
        const int32_t nw = words[size_t(sg)];
        if (off < 0 || nw < 0 || int64_t(off) + nw > int64_t(sd.prog.size()))
            return "streamed program outside the table";
        const size_t S = size_t(sd.slots);
        std::vector<int64_t> slot(S, -1), pend(S, -1);   // term; its load (number)
        std::vector<int64_t> ld_of(n, -1);               // last load of a row
        std::vector<char> st_pend(n, 0);                 // a store to a row in flight
        int64_t seq = 0, done = 0;  // loads issued; those before `done` finished
        auto read = [&](uint32_t sl, int64_t& t) -> const char* {
            if (sl >= S) return "streamed slot out of range";
            if (pend[sl] >= done) return "streamed slot read while its load may be in flight";
            if (slot[sl] < 0) return "streamed slot read before it holds a value";
            t = slot[sl];
            return nullptr;
        };
        const uint32_t* sp = sd.prog.data() + off;
        for (int32_t c0 = 0; c0 < nw; c0 += 64) {
            const int32_t m = std::min(64, nw - c0);
            int32_t c = 0;
            while (c < m) {
                const uint32_t h = sp[c0 + c], op = h & 0xFF;
                const uint32_t b1 = (h >> 8) & 0xFF, b2 = (h >> 16) & 0xFF, b3 = h >> 24;
                if (op == 0) {
                    for (int32_t j = c; j < m; ++j)
                        if (sp[c0 + j]) return "streamed chunk padding not zero";
                    break;
                }
                int32_t len = 1;
                if (op == kResAdd2 || op == kResFold) {
                    std::vector<uint32_t> src;
                    uint32_t d;
                    if (op == kResAdd2) {
                        src = {b1, b2};
                        d = b3;
                    } else {
                        len = 1 + int32_t(b1 + 3) / 4;
                        if (b1 < 2 || b3 || c + len > m) return "streamed fold malformed or across a chunk";
                        for (uint32_t i = 0; i < b1; ++i)
                            src.push_back((sp[c0 + c + 1 + i / 4] >> (8 * (i % 4))) & 0xFF);
                        d = b2;
                    }
                    std::vector<int64_t> v;
                    for (uint32_t r : src) {
                        int64_t t;
                        if (const char* e = read(r, t)) return e;
                        v.push_back(t);
                    }
                    if (d >= S) return "streamed slot out of range";
                    if (pend[d] >= done) return "streamed fold into a slot whose load may be in flight";
                    slot[d] = fold(v);
                    pend[d] = -1;
                } else if (op == kResLoad) {
                    len = 1 + int32_t(b1);
                    if (b1 < 1 || b2 || b3 || c + len > m) return "streamed load malformed or across a chunk";
                    for (uint32_t i = 0; i < b1; ++i) {
                        const uint32_t x = sp[c0 + c + 1 + i], sl = x & 0xFF, b = x >> 8;
                        if (sl >= S || b >= n) return "streamed load out of range";
                        if (pend[sl] >= done) return "streamed load into a slot whose load may be in flight";
                        if (st_pend[b]) return "streamed load of a row whose store may be in flight";
                        slot[sl] = hbm[b];
                        pend[sl] = ld_of[b] = seq++;
                    }
                } else if (op == kResWait) {
                    if (b2 || b3) return "streamed wait malformed";
                    done = std::max(done, seq - int64_t(b1));
                    if (b1 == 0) std::fill(st_pend.begin(), st_pend.end(), char(0));
                } else if (op == kResPut) {
                    len = 1 + int32_t(b1 + 1) / 2;
                    if (b1 < 1 || b3 || c + len > m) return "streamed store malformed or across a chunk";
                    int64_t t;
                    if (const char* e = read(b2, t)) return e;
                    for (uint32_t i = 0; i < b1; ++i) {
                        const uint32_t x = sp[c0 + c + 1 + i / 2];
                        const uint32_t b = i % 2 ? x >> 16 : x & 0xFFFF;
                        if (b >= n) return "streamed store out of range";
                        if (ld_of[b] >= done) return "streamed store to a row whose load may be in flight";
                        hbm[b] = t;
                        st_pend[b] = 1;
                    }
                    if (b1 % 2 && (sp[c0 + c + len - 1] >> 16)) return "streamed store padding not zero";
                } else {
                    return "streamed record with an unknown opcode";
                }
                c += len;
            }
        }
        for (size_t b = 0; b < n; ++b)
            if (hbm[b] != want[b]) return "streamed result differs from the phases' steps";
    }
    for (int64_t i = 0; i < sd.nunits; ++i) {
        const ResUnit& u = sd.runits[size_t(i)];
        const int2 e = sd.tiles[size_t(i)];
        const size_t sg = size_t(e.x);
        const int64_t lo = sd.cuts[sg] + int64_t(e.y) * sd.tile_elems;
        const int64_t nv = std::min(sd.tile_elems, sd.cuts[sg + 1] - lo) / VEC;
        if (u.lo != lo || u.nv != nv || nv < 1 || nv > 64) return "streamed unit tile";
        if (u.load || u.store || u.alias != -1) return "streamed unit with row masks";
        if (u.off != sd.rec_off[sg] || u.nw != words[sg] || u.nw > sd.max_nw)
            return "streamed unit program";
    }
    return "";
}

// Host-side check of the executed phases and the launch tiling (no GPU):
// every executed phase is free of hazards, and walking every wave tile of
// every launch with the kernel's own index helpers covers each step exactly
// once, in bounds, with 16-byte aligned vector parts (the padding entries of
// a tile table excepted, which the kernel skips).  In a split launch the
// waves of a workgroup share one tile, and their shares of a step's
// destinations cover each destination once, the ones among the step's
// sources (stored after the barrier) last.  An affinity table puts every
// tile on the XCD (workgroup id modulo kNumXCDs) that xcd_of names.
AR_EXPORT ar_status ar_debug_check_tiling(ar_plan* plan, int32_t vecok,
                                          char* msg, int64_t msglen) {
    clear_error();
    auto bad = [&](const std::string& m) {
        if (msg && msglen > 0) {
            std::strncpy(msg, m.c_str(), size_t(msglen - 1));
            msg[msglen - 1] = 0;
        }
        return fail(AR_ERR_INTERNAL, m);
    };
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    try {
        ExecState* ex = exec_state(*plan);
        std::string why;
        if (!exec_phases_hazard_free(ex->phases, plan->n, why)) return bad(why);
        const int64_t VEC = 16 / plan->esize;
        std::vector<std::vector<std::pair<int64_t, int64_t>>> cover(ex->hsteps.size());
        std::vector<char> launched(ex->hsteps.size(), 0);
        for (const LaunchDesc& L : ex->launches) {
            if (L.nunits <= 0) return bad("launch without work units");
            const int64_t blocks = (L.nunits + L.wpb - 1) / L.wpb;
            if (blocks > kMaxBlocks) return bad("grid too large");
            if (L.wpb != (L.dsplit > 1 ? kSplitWaves : kcfg(L.kern_k).WPB))
                return bad("block size differs from the kernel's");
            if (L.rt_group < 1 || L.rt_group > kRtGroup) return bad("source group out of range");
            if (L.tile_elems % (64 * VEC) != 0) return bad("tile not a multiple of a wave vector");
            if (L.dsplit < 1 || (L.dsplit > 1 && (L.dsplit != L.wpb || L.nunits % L.dsplit)))
                return bad("split launch not one tile per workgroup");
            const int2* tiles = L.tile_off >= 0 ? ex->htiles.data() + L.tile_off : nullptr;
            if (tiles && L.tile_off + L.nunits / L.dsplit > int64_t(ex->htiles.size()))
                return bad("tile table overrun");
            for (int64_t j = 0; j < L.count; ++j) launched[size_t(L.first + j)] = 1;
            for (int64_t unit = 0; unit < blocks * L.wpb; ++unit) {
                if (unit >= L.nunits) continue;  // the kernel returns here
                const int64_t tile = L.dsplit > 1 ? unit / L.dsplit : unit;
                const int part = int(unit - tile * L.dsplit);
                int64_t s, t;
                unit_tile(tile, tiles, L.tiles_per_step, s, t);
                if (tiles && s == -1 && t == 0) continue;  // padding entry: the kernel skips it
                if (s < 0 || s >= L.count || t < 0) return bad("unit maps outside the launch");
                const DevStep& st = ex->hsteps[size_t(L.first + s)];
                if (L.affinity && !tiles) return bad("affinity launch without a tile table");
                if (L.affinity &&
                    xcd_of(std::max((st.begin & ~(VEC - 1)) + t * L.tile_elems, st.begin),
                           plan->N) != (unit / L.wpb) % kNumXCDs)
                    return bad("tile not on the XCD of its position");
                if (st.k < 1 || st.src_off < 0 ||
                    int64_t(st.src_off) + st.k > int64_t(ex->hidx.size()))
                    return bad("source list out of range");
                if (L.kern_k != 0 && st.k != L.kern_k) return bad("source count differs from the kernel's");
                for (int32_t q = 0; q < st.k; ++q) {
                    const int32_t src = ex->hidx[size_t(st.src_off + q)];
                    if (src < 0 || src >= plan->n) return bad("source index out of range");
                }
                if (st.ndst < 1 || st.dst_off < 0 ||
                    int64_t(st.dst_off) + st.ndst > int64_t(ex->hidx.size()))
                    return bad("destination list out of range");
                for (int32_t q = 0; q < st.ndst; ++q) {
                    const int32_t dst = ex->hidx[size_t(st.dst_off + q)];
                    if (dst < 0 || dst >= plan->n) return bad("destination index out of range");
                    bool is_src = false;
                    for (int32_t j = 0; j < st.k; ++j)
                        is_src = is_src || ex->hidx[size_t(st.src_off + j)] == dst;
                    if (is_src != (q >= st.nfree))
                        return bad("destinations among the sources not last");
                }
                if (L.dsplit > 1 && part == L.dsplit - 1) {
                    // the parts' shares tile [0, nfree) and [nfree, ndst)
                    int fa = 0, ga = 0;
                    for (int pp = 0; pp < L.dsplit; ++pp) {
                        int a, b;
                        split_share(st.nfree, pp, L.dsplit, a, b);
                        if (a != fa || b < a) return bad("destination shares not contiguous");
                        fa = b;
                        split_share(st.ndst - st.nfree, pp, L.dsplit, a, b);
                        if (a != ga || b < a) return bad("destination shares not contiguous");
                        ga = b;
                    }
                    if (fa != st.nfree || ga != st.ndst - st.nfree)
                        return bad("destination shares do not cover the step");
                }
                const TileSpan sp = tile_span(st.begin, st.end, t, L.tile_elems, VEC, vecok != 0);
                if (sp.lo >= sp.hi) continue;
                if (sp.lo < st.begin || sp.hi > st.end || st.begin < 0 || st.end > plan->N)
                    return bad("tile outside its step");
                if (!(sp.lo <= sp.vlo && sp.vlo <= sp.vhi && sp.vhi <= sp.hi))
                    return bad("vector part outside its tile");
                if (sp.vhi > sp.vlo && (!vecok || sp.vlo % VEC || sp.vhi % VEC))
                    return bad("misaligned vector part");
                if (sp.vlo - sp.lo >= VEC || (sp.vhi > sp.vlo && sp.hi - sp.vhi >= VEC))
                    if (sp.vhi > sp.vlo) return bad("head or tail longer than a vector");
                if (part == 0) cover[size_t(L.first + s)].push_back({sp.lo, sp.hi});
            }
        }
        // step records: inside the record area, disjoint, long enough for
        // the step's pointers, at the launch's stride
        {
            if (ex->rec_of.size() != ex->hsteps.size()) return bad("a step without a record");
            std::vector<std::pair<int64_t, int64_t>> iv;
            for (size_t i = 0; i < ex->hsteps.size(); ++i) {
                const DevStep& st = ex->hsteps[i];
                const int64_t o = ex->rec_of[i];
                if (o < 0 || o + kRecHead + st.k + st.ndst > ex->rec_words)
                    return bad("step record outside the record area");
                iv.push_back({o, o + kRecHead + st.k + st.ndst});
            }
            std::sort(iv.begin(), iv.end());
            for (size_t i = 1; i < iv.size(); ++i)
                if (iv[i].first < iv[i - 1].second) return bad("step records overlap");
            for (const LaunchDesc& L : ex->launches)
                for (int64_t j = 0; j < L.count; ++j) {
                    const DevStep& st = ex->hsteps[size_t(L.first + j)];
                    if (ex->rec_of[size_t(L.first + j)] != L.rec_off + j * L.rec_stride)
                        return bad("record not at the launch's stride");
                    if (L.rec_stride < kRecHead + st.k + st.ndst || L.rec_off % 2 || L.rec_stride % 2)
                        return bad("record stride too short or misaligned");
                }
        }
        for (size_t i = 0; i < ex->hsteps.size(); ++i) {
            const DevStep& st = ex->hsteps[i];
            auto& c = cover[i];
            if (st.end > st.begin && !launched[i]) return bad("step never launched");
            std::sort(c.begin(), c.end());
            int64_t at = st.begin;
            for (auto& iv : c) {
                if (iv.first != at) return bad("gap or overlap in step " + std::to_string(i));
                at = iv.second;
            }
            if (st.end > st.begin && at != st.end)
                return bad("step " + std::to_string(i) + " not covered to its end");
        }
        // sliced launches: the runs are disjoint and in order, every stage
        // names a launch or a slice, every launch of a phase outside the
        // slices runs once; a slice's tiles cover each segment some step of
        // its phases covers exactly once with aligned vectors, and each
        // (phase, segment) lists exactly the steps of that phase covering the
        // segment
        {
            std::vector<int32_t> slice_of(ex->phases.size(), -1);
            int32_t prev_end = 0;
            for (size_t k = 0; k < ex->slices.size(); ++k) {
                const SliceDesc& sd = ex->slices[k];
                if (!sd.ok || sd.nphases < 1 || sd.p0 < prev_end ||
                    sd.p0 + sd.nphases > int32_t(ex->phases.size()))
                    return bad("slice phase range out of order");
                prev_end = sd.p0 + sd.nphases;
                for (int32_t q = sd.p0; q < prev_end; ++q) slice_of[size_t(q)] = int32_t(k);
            }
            std::vector<int32_t> runs_of(ex->launches.size(), 0), seen(ex->slices.size(), 0);
            for (const Stage& stg : ex->stages) {
                if (stg.slice >= 0) {
                    if (stg.slice >= int32_t(ex->slices.size())) return bad("stage names no slice");
                    ++seen[size_t(stg.slice)];
                } else {
                    if (stg.launch < 0 || stg.launch >= int32_t(ex->launches.size()))
                        return bad("stage names no launch");
                    ++runs_of[size_t(stg.launch)];
                }
            }
            for (size_t k = 0; k < ex->slices.size(); ++k)
                if (seen[k] != 1) return bad("slice not run exactly once");
            for (size_t li = 0; li < ex->launches.size(); ++li)
                if (runs_of[li] != (slice_of[size_t(ex->launches[li].xphase)] < 0 ? 1 : 0))
                    return bad("phase launch not run exactly once outside the slices");
        }
        for (const SliceDesc& sd : ex->slices) {
            std::vector<std::vector<std::pair<int64_t, int64_t>>> sc(size_t(sd.nseg));
            for (int64_t u = 0; u < sd.nunits; ++u) {
                const int2 e = sd.tiles[size_t(u)];
                if (e.x < 0 || e.x >= sd.nseg || e.y < 0) return bad("slice tile out of range");
                const int64_t lo = sd.cuts[size_t(e.x)] + int64_t(e.y) * sd.tile_elems;
                const int64_t hi = std::min(sd.cuts[size_t(e.x) + 1], lo + sd.tile_elems);
                if (lo >= hi || lo % VEC || hi % VEC) return bad("slice tile empty or misaligned");
                if ((hi - lo) / VEC > (sd.resident ? 64 : 64 * kSliceU)) return bad("slice tile too long");
                sc[size_t(e.x)].push_back({lo, hi});
            }
            if (int64_t(sd.sched_off.size()) != int64_t(sd.nphases) * sd.nseg + 1)
                return bad("schedule offsets of the wrong size");
            for (int32_t sg = 0; sg < sd.nseg; ++sg) {
                bool covered = false;
                for (int32_t q = 0; q < sd.nphases; ++q) {
                    const size_t o = size_t(q) * size_t(sd.nseg) + size_t(sg);
                    if (sd.sched_off[o + 1] > sd.sched_off[o]) covered = true;
                }
                auto& c = sc[size_t(sg)];
                if (!covered) {
                    if (!c.empty()) return bad("slice tiles on a segment no step covers");
                    continue;
                }
                std::sort(c.begin(), c.end());
                int64_t at = sd.cuts[size_t(sg)];
                for (auto& iv : c) {
                    if (iv.first != at) return bad("slice tiles leave a gap or overlap");
                    at = iv.second;
                }
                if (at != sd.cuts[size_t(sg) + 1]) return bad("slice tiles do not cover a segment");
            }
            for (int32_t q = 0; q < sd.nphases; ++q) {
                const XPhase& xp = ex->phases[size_t(sd.p0 + q)];
                for (int32_t sg = 0; sg < sd.nseg; ++sg) {
                    std::vector<int32_t> want, got;
                    for (size_t i = 0; i < xp.steps.size(); ++i) {
                        const XStep& x = xp.steps[i];
                        if (x.end <= x.begin) continue;
                        if (x.begin <= sd.cuts[size_t(sg)] && sd.cuts[size_t(sg) + 1] <= x.end)
                            want.push_back(int32_t(
                                ex->rec_of[size_t(ex->dev_of[size_t(sd.p0 + q)][i])]));
                        else if (x.begin < sd.cuts[size_t(sg) + 1] && sd.cuts[size_t(sg)] < x.end)
                            return bad("a step cuts a segment");
                    }
                    const size_t o = size_t(q) * size_t(sd.nseg) + size_t(sg);
                    for (int32_t i = sd.sched_off[o]; i < sd.sched_off[o + 1]; ++i)
                        got.push_back(sd.sched[size_t(i)]);
                    std::sort(want.begin(), want.end());
                    std::sort(got.begin(), got.end());
                    if (want != got) return bad("schedule differs from the steps of a phase");
                }
            }
            if (sd.streamed) {
                const std::string e = check_streamed(*plan, *ex, sd);
                if (!e.empty()) return bad(e);
            } else if (sd.resident) {
                // per segment: running its records symbolically (each value a
                // term: an input row, an unordered 2-operand add, the rounding
                // at the end of a fold) gives, for every row it stores, the
                // term the executed steps give (phase by phase, each phase
                // reading the state it started with), and leaves every other
                // row's term the input; no record reads a row that is neither
                // loaded nor written before, no record crosses a 64-word chunk;
                // per unit: its tile, and the rows to load (read before
                // written) and to store (written) of its segment
                if (plan->n > kResMaxN) return bad("resident launch with too many buffers");
                if (sd.res_waves != 1 && sd.res_waves != 4) return bad("resident workgroup size");
                if (int64_t(sd.runits.size()) != sd.nunits || int64_t(sd.tiles.size()) != sd.nunits ||
                    int64_t(sd.rec_off.size()) != sd.nseg)
                    return bad("resident table sizes");
                std::vector<uint64_t> wload(size_t(sd.nseg), 0), wstore(size_t(sd.nseg), 0);
                std::vector<int32_t> words(size_t(sd.nseg), 0);
                for (int32_t sg = 0; sg < sd.nseg; ++sg) {
                    std::map<std::tuple<int, int64_t, int64_t>, int64_t> terms;
                    auto term = [&](int kind, int64_t x, int64_t y) {
                        if (kind == 1 && x > y) std::swap(x, y);  // add: unordered
                        auto it = terms.emplace(std::make_tuple(kind, x, y), int64_t(terms.size())).first;
                        return it->second;
                    };
                    auto fold = [&](const std::vector<int64_t>& v) {  // k >= 1 operand terms
                        if (v.size() == 1) return v[0];
                        int64_t t = v[0];
                        for (size_t j = 1; j < v.size(); ++j) t = term(1, t, v[j]);
                        return term(2, t, 0);
                    };
                    const size_t n = size_t(plan->n);
                    std::vector<int64_t> want(n), input(n);
                    for (size_t b = 0; b < n; ++b) want[b] = input[b] = term(0, int64_t(b), 0);
                    uint64_t seen = 0;
                    bool covered = false;
                    for (int32_t q = 0; q < sd.nphases; ++q) {
                        std::vector<std::pair<int32_t, int64_t>> outs;
                        for (const XStep& x : ex->phases[size_t(sd.p0 + q)].steps) {
                            if (!(x.end > x.begin && x.begin <= sd.cuts[size_t(sg)] &&
                                  sd.cuts[size_t(sg) + 1] <= x.end))
                                continue;
                            covered = true;
                            std::vector<int64_t> v;
                            for (int32_t b : x.srcs) {
                                v.push_back(want[size_t(b)]);
                                if (!(seen >> b & 1)) wload[size_t(sg)] |= uint64_t(1) << b;
                            }
                            for (int32_t b : x.srcs) seen |= uint64_t(1) << b;
                            const int64_t t = fold(v);
                            for (int32_t b : x.dsts) {
                                outs.push_back({b, t});
                                seen |= uint64_t(1) << b;
                                wstore[size_t(sg)] |= uint64_t(1) << b;
                            }
                        }
                        for (const auto& o : outs) want[size_t(o.first)] = o.second;
                    }
                    const int32_t off = sd.rec_off[size_t(sg)];
                    if (!covered) {
                        if (off != -1) return bad("resident records on an idle segment");
                        continue;
                    }
                    // the segment's unit records give its record count
                    int32_t nw = -1, aoff = -1;
                    for (int64_t i = 0; i < sd.nunits; ++i)
                        if (sd.tiles[size_t(i)].x == sg) {
                            nw = sd.runits[size_t(i)].nw;
                            aoff = sd.runits[size_t(i)].alias;
                            break;
                        }
                    if (off < 0 || nw < 1 || int64_t(off) + nw > int64_t(sd.prog.size()))
                        return bad("resident records outside the table");
                    // the row each stored buffer takes its value from
                    std::vector<uint32_t> src_row(n);
                    for (size_t b = 0; b < n; ++b) src_row[b] = uint32_t(b);
                    if (aoff >= 0) {
                        if (int64_t(aoff) + 16 > int64_t(sd.prog.size())) return bad("resident alias table outside the table");
                        for (size_t b = 0; b < 64; ++b) {
                            const uint32_t a = (sd.prog[size_t(aoff) + b / 4] >> (8 * (b % 4))) & 0xFF;
                            if (a == 0xFF) continue;
                            if (b >= n || a >= n || !(wstore[size_t(sg)] >> b & 1))
                                return bad("resident alias entry out of range or not stored");
                            src_row[b] = a;
                        }
                    }
                    std::vector<int64_t> have(n, -1);
                    for (size_t b = 0; b < n; ++b)
                        if (wload[size_t(sg)] >> b & 1) have[b] = input[b];
                    auto get = [&](uint32_t r, int64_t& t) {
                        if (r >= n || have[r] < 0) return false;
                        t = have[r];
                        return true;
                    };
                    int64_t last = -1;  // the previous record's result
                    const uint32_t* sp = sd.prog.data() + off;
                    for (int32_t c0 = 0; c0 < nw; c0 += 64) {
                        const int32_t m = std::min(64, nw - c0);
                        int32_t c = 0;
                        while (c < m) {
                            const uint32_t h = sp[c0 + c];
                            const uint32_t op = h & 0xFF;
                            if (op == 0) {
                                for (int32_t j = c; j < m; ++j)
                                    if (sp[c0 + j]) return bad("resident chunk padding not zero");
                                break;
                            }
                            auto row = [&](int32_t i) {  // row byte i after the header
                                return (sp[c0 + c + 1 + i / 4] >> (8 * (i % 4))) & 0xFF;
                            };
                            std::vector<uint32_t> dsts;
                            int64_t t = 0, y = 0;
                            int32_t len = 1;
                            if (op == kResAdd2 || op == kResCopy) {
                                const uint32_t r0 = (h >> 8) & 0xFF, r1 = (h >> 16) & 0xFF;
                                if (op == kResCopy && r1 != r0) return bad("resident copy record malformed");
                                if (!get(r0, t)) return bad("resident record reads an unloaded row");
                                if (op == kResAdd2) {
                                    if (!get(r1, y)) return bad("resident record reads an unloaded row");
                                    t = fold({t, y});
                                }
                                dsts.push_back(h >> 24);
                            } else if (op == kResChain || op == kResFold) {
                                const int32_t k = int32_t((h >> 8) & 0xFF);
                                len = 1 + (k + 3) / 4;
                                if (k < 1 || (op == kResFold && (k < 2 || (h >> 24))) || c + len > m)
                                    return bad("resident record malformed or across a chunk");
                                std::vector<int64_t> v;
                                if (op == kResChain) {
                                    if (!get((h >> 16) & 0xFF, t)) return bad("resident chain reads an unloaded row");
                                    for (int32_t i = 0; i < k; ++i) {
                                        if (!get(row(i), y)) return bad("resident chain reads an unloaded row");
                                        t = fold({t, y});
                                    }
                                    dsts.push_back(h >> 24);
                                } else {
                                    for (int32_t i = 0; i < k; ++i) {
                                        if (!get(row(i), y)) return bad("resident fold reads an unloaded row");
                                        v.push_back(y);
                                    }
                                    t = fold(v);
                                    dsts.push_back((h >> 16) & 0xFF);
                                }
                            } else if (op == kResStore) {
                                const int32_t nd = int32_t((h >> 8) & 0xFF);
                                len = 1 + nd / 4;
                                if (nd < 4 || nd % 4 || (h >> 16) || c + len > m)
                                    return bad("resident store record malformed or across a chunk");
                                if (last < 0) return bad("resident store without a result before it");
                                t = last;
                                for (int32_t i = 0; i < nd; ++i) dsts.push_back(row(i));
                            } else {
                                return bad("resident record with an unknown opcode");
                            }
                            for (uint32_t d : dsts) {
                                if (d >= n) return bad("resident row out of range");
                                have[d] = t;
                            }
                            last = t;
                            c += len;
                        }
                    }
                    for (size_t b = 0; b < n; ++b) {
                        if (wstore[size_t(sg)] >> b & 1) {
                            if (have[src_row[b]] != want[b])
                                return bad("resident result differs from the phases' steps");
                        } else if (want[b] != input[b]) {
                            return bad("resident launch leaves a written row unstored");
                        }
                    }
                    words[size_t(sg)] = nw;
                }
                std::vector<int64_t> first_unit(size_t(sd.nseg), -1);
                for (int64_t i = sd.nunits; i-- > 0;) first_unit[size_t(sd.tiles[size_t(i)].x)] = i;
                for (int64_t i = 0; i < sd.nunits; ++i) {
                    const ResUnit& u = sd.runits[size_t(i)];
                    const int2 e = sd.tiles[size_t(i)];
                    const size_t sg = size_t(e.x);
                    const int64_t lo = sd.cuts[sg] + int64_t(e.y) * sd.tile_elems;
                    const int64_t nv = std::min(sd.tile_elems, sd.cuts[sg + 1] - lo) / VEC;
                    if (u.lo != lo || u.nv != nv || nv < 1 || nv > 64) return bad("resident unit tile");
                    if (u.load != wload[sg] || u.store != wstore[sg]) return bad("resident unit rows");
                    if (u.off != sd.rec_off[sg] || u.nw != words[sg] ||
                        int64_t(u.off) + u.nw > int64_t(sd.prog.size()))
                        return bad("resident unit records");
                    if (u.alias != sd.runits[size_t(first_unit[sg])].alias) return bad("resident unit alias table");
                }
            }
            // every step of the slice's phases lies inside the segments
            for (int32_t q = 0; q < sd.nphases; ++q)
                for (const XStep& x : ex->phases[size_t(sd.p0 + q)].steps)
                    if (x.end > x.begin &&
                        (!std::binary_search(sd.cuts.begin(), sd.cuts.end(), x.begin) ||
                         !std::binary_search(sd.cuts.begin(), sd.cuts.end(), x.end)))
                        return bad("a step boundary is not a segment boundary");
        }
        if (msg && msglen > 0) msg[0] = 0;
        return AR_OK;
    } catch (const std::exception& e) {
        return bad(e.what());
    }
}

AR_EXPORT ar_status ar_debug_exec_steps(ar_plan* plan, int64_t step_cap, int32_t* phase,
                                        int64_t* begin, int64_t* end, int32_t* nsrc,
                                        int32_t* ndst, int64_t idx_cap, int32_t* idx,
                                        int64_t* count, int64_t* idx_count) {
    clear_error();
    if (!plan || !count || !idx_count) return fail(AR_ERR_INVALID_ARG, "NULL argument");
    try {
        const ExecState* ex = exec_state(*plan);
        int64_t c = 0, ic = 0;
        for (size_t q = 0; q < ex->phases.size(); ++q)
            for (const XStep& x : ex->phases[q].steps) {
                if (c < step_cap) {
                    if (phase) phase[c] = int32_t(q);
                    if (begin) begin[c] = x.begin;
                    if (end) end[c] = x.end;
                    if (nsrc) nsrc[c] = int32_t(x.srcs.size());
                    if (ndst) ndst[c] = int32_t(x.dsts.size());
                }
                ++c;
                for (int32_t v : x.srcs) {
                    if (idx && ic < idx_cap) idx[ic] = v;
                    ++ic;
                }
                for (int32_t v : x.dsts) {
                    if (idx && ic < idx_cap) idx[ic] = v;
                    ++ic;
                }
            }
        *count = c;
        *idx_count = ic;
        return AR_OK;
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}

AR_EXPORT ar_status ar_debug_resident(ar_plan* plan, int32_t stage, int64_t* info,
                                      int64_t* units, uint32_t* prog) {
    clear_error();
    if (!plan || !info) return fail(AR_ERR_INVALID_ARG, "NULL argument");
    try {
        const ExecState* ex = exec_state(*plan);
        if (stage < 0 || stage >= int32_t(ex->stages.size()) || ex->stages[size_t(stage)].slice < 0 ||
            !ex->slices[size_t(ex->stages[size_t(stage)].slice)].resident)
            return fail(AR_ERR_INVALID_ARG, "not a resident launch");
        const SliceDesc& sd = ex->slices[size_t(ex->stages[size_t(stage)].slice)];
        info[0] = sd.p0;
        info[1] = sd.nphases;
        info[2] = sd.nunits;
        info[3] = int64_t(sd.prog.size());
        info[4] = sd.streamed ? sd.slots : 0;
        if (units)
            for (size_t i = 0; i < sd.runits.size(); ++i) {
                const ResUnit& u = sd.runits[i];
                int64_t* o = units + 7 * i;
                o[0] = u.lo;
                o[1] = int64_t(u.load);
                o[2] = int64_t(u.store);
                o[3] = u.nv;
                o[4] = u.off;
                o[5] = u.nw;
                o[6] = u.alias;
            }
        if (prog) std::copy(sd.prog.begin(), sd.prog.end(), prog);
        return AR_OK;
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}

AR_EXPORT ar_status ar_debug_launch_desc(ar_plan* plan, int32_t stage, int64_t* out) {
    clear_error();
    if (!plan || !out) return fail(AR_ERR_INVALID_ARG, "NULL argument");
    try {
        const ExecState* ex = exec_state(*plan);
        if (stage < 0 || stage >= int32_t(ex->stages.size()))
            return fail(AR_ERR_INVALID_ARG, "launch index out of range");
        const Stage stg = ex->stages[size_t(stage)];
        if (stg.slice >= 0) return fail(AR_ERR_INVALID_ARG, "a sliced launch");
        const LaunchDesc& L = ex->launches[size_t(stg.launch)];
        out[0] = L.kern_k;
        out[1] = L.cm;
        out[2] = L.tile_elems;
        out[3] = L.nunits;
        out[4] = L.wpb;
        out[5] = L.tile_off >= 0 ? 1 : 0;
        out[6] = L.rt_group;
        out[7] = L.dsplit;
        out[8] = L.affinity;
        out[9] = L.wide;
        return AR_OK;
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}
