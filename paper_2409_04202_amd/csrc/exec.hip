// Executor: turns a plan's phases into batched kernel launches on a HIP
// stream, plus the timing API.
//
// Per phase, the steps are grouped by source count k (copies are k = 1) and
// each group becomes one launch of phase_kernel<dtype, k, aligned>; the
// built-in plans have one group per phase.  Kernels read each step as a
// record holding its range and its resolved buffer pointers (StepHead);
// the records of a buffer set are built on the host and uploaded once, and a
// small per-plan cache keeps them per device, so repeated executes on the
// same buffers launch kernels only.  The sliced-launch tables are uploaded
// on the first execute on a device.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <map>
#include <memory>
#include <tuple>
#include <new>
#include <string>
#include <vector>

#include "ar_debug.h"
#include "internal.hpp"
#include "kernels.hpp"

namespace arp {

namespace {

constexpr int kCache = 4;               // buffer sets whose step records are kept per device
constexpr int64_t kMinUnits = 2048;     // shrink tiles until a launch has this many
constexpr int64_t kMaxBlocks = int64_t(1) << 24;
// Cache policy per launch (measured on MI355X).  Launches moving less than
// kNtBytes keep everything cached.  Larger ones load nontemporally unless a
// source range is read by more than one step of the launch (then the repeated
// reads hit the cache), and store nontemporally unless the next phase reads
// what they write and it is at most kKeepBytes, small enough to stay in the
// 256 MiB last-level cache until then.
constexpr int64_t kNtBytes = int64_t(64) << 20;
constexpr int64_t kKeepBytes = int64_t(256) << 20;
// The step rewrites (multicast, reduce-then-broadcast) pay off where they
// remove a launch from a short phase, add at most one extra destination, or
// take over copies that read every range once (their reads are saved; a
// 2-source fold storing to 8 destinations streams at 5.0 TB/s); a step
// storing to many destinations over a large range is slower than plain
// copies whose repeated reads hit the cache.  A rewrite is applied when its
// step ends with at most kFuseDst destinations, the copies it takes over
// move at most kFuseBytes (2 * len * e each), or (reduce-then-broadcast) no
// two of those copies read the same range.
constexpr int32_t kFuseDst = 2;
constexpr int64_t kFuseBytes = int64_t(256) << 20;
// Automatic choice of sliced launches (AR_OPT_SLICE = 2).  A run of
// consecutive executed phases may become one sliced launch when every phase
// in it writes at most kKeepBytes (what one phase hands to the next would
// stay in the last-level cache with phase launches as well) and moves at most
// kSliceMaxBytes.  The runs are chosen by dynamic programming over the phases
// with a cost model fitted to MI355X measurements (back-to-back launches, no
// events between them):
//  * a phase launch costs kLaunchNs plus its bytes at kBytesPerNs;
//  * a sliced launch costs kLaunchNs plus, per phase, the largest of its
//    dependent chain, its read time and its write time.  The chain is the
//    most steps covering one element position, which a wavefront runs one
//    after the other, at kStepNs + k * kStepNsPerSrc{F32,BF16} +
//    d * kStepNsPerDst each (k, d = the phase's largest source and
//    destination counts); reads and writes go at kBytesPerNs, the reads
//    stretched by kMinSliceWaves / waves when the slice has fewer wave tiles
//    than that (too few loads in flight to reach full bandwidth).
constexpr double kLaunchNs = 3000.0;
constexpr double kBytesPerNs = 5500.0;
constexpr double kStepNs = 350.0;
constexpr double kStepNsPerSrcF32 = 120.0;
constexpr double kStepNsPerSrcBF16 = 190.0;
constexpr double kStepNsPerDst = 15.0;
constexpr double kMinSliceWaves = 256.0;
constexpr int64_t kSliceMaxBytes = int64_t(512) << 20;

struct LaunchDesc {
    int32_t phase;
    int32_t xphase;          // executed phase
    int32_t kern_k;          // template K (0 = runtime source count)
    int64_t first;           // first entry of the step table (hsteps)
    int64_t count;           // steps in this launch
    int64_t tile_elems;
    int64_t tiles_per_step;  // arithmetic mapping
    int64_t nunits;          // wave tiles
    int64_t tile_off;        // -1, or first entry of the device tile table
    int32_t wpb;             // wavefronts per block
    int32_t cm;              // cache mode: bit 0 NT loads, bit 1 NT stores
    int32_t max_dst;         // most destinations of a step
    int64_t bytes;           // (k + destinations) * len * e over the steps
    int64_t rec_off;         // first word of its steps' records
    int64_t rec_stride;      // words per record
};

// The step records of one buffer set on one device.
struct PtrEntry {
    std::vector<void*> key;
    uint64_t* dev = nullptr;     // records, device
    uint64_t* pinned = nullptr;  // staging for their upload
    hipEvent_t done = nullptr;
    uint64_t stamp = 0;
    bool valid = false;
    bool aligned = false;
};

struct DevState {
    int device = -1;
    int2* tiles = nullptr;
    int64_t* cuts = nullptr;     // sliced launch tables, all slices concatenated
    int32_t* sched_off = nullptr;
    int32_t* sched = nullptr;
    int2* stiles = nullptr;
    PtrEntry cache[kCache];
    uint64_t clock = 0;
};

int kernel_k(int32_t k) {
    switch (k) {
        case 1: case 2: case 3: case 4: case 8: case 16: return k;
        default: return 0;
    }
}

std::string hip_msg(const char* what, hipError_t e) {
    return std::string(what) + ": " + hipGetErrorName(e) + " (" +
           hipGetErrorString(e) + ")";
}

}  // namespace

// An executed step (host form): fold `srcs` over [begin, end) and store the
// result into every destination.  Plan steps map one to one onto executed
// steps unless the rewrites below merge them.
struct XStep {
    int64_t begin, end;
    std::vector<int32_t> srcs;
    std::vector<int32_t> dsts;
};

struct XPhase {
    int32_t plan_phase;  // phase of the plan these steps come from
    std::vector<XStep> steps;
};

// A sliced launch runs executed phases [p0, p0 + nphases): segments are the
// element ranges between consecutive boundaries of those phases' steps;
// sched lists, per (phase of the slice, segment), the word offsets of the
// records of the steps covering that segment; tiles maps each wavefront to (segment, tile within the
// segment), over the segments some step of the slice covers.
struct SliceDesc {
    bool ok = false;
    std::string why;             // why the phases cannot run sliced
    int32_t p0 = 0, nphases = 0, nseg = 0;
    int64_t tile_elems = 0, nunits = 0, bytes = 0, nsteps = 0;
    int64_t chain = 0;           // sum over phases of the most steps on a segment
    int32_t max_k = 0, max_dst = 0;
    std::vector<int64_t> cuts;
    std::vector<int32_t> sched_off, sched;
    std::vector<int2> tiles;
    // offsets of this slice's tables in the concatenated device tables
    int64_t cuts_base = 0, soff_base = 0, sched_base = 0, tiles_base = 0;
};

// One launch of an execution: a sliced launch (slice >= 0) or the phase
// launch `launch`.
struct Stage {
    int32_t slice;
    int32_t launch;
};

struct ExecState {
    std::vector<XPhase> phases;  // executed phases, after the rewrites
    std::vector<LaunchDesc> launches;
    std::vector<DevStep> hsteps;
    std::vector<int32_t> hidx;   // source and destination indices
    std::vector<int2> htiles;
    std::vector<std::vector<int32_t>> dev_of;  // [phase][step] -> hsteps index
    std::vector<int64_t> rec_of; // hsteps index -> first word of its record
    int64_t rec_words = 0;       // words of all records
    std::vector<SliceDesc> slices;
    std::vector<Stage> stages;   // the launches for 16-byte aligned buffers
    std::vector<DevState*> dev;  // indexed by device ordinal
};

// Every (buffer, range) a phase touches, with the step touching it; answers
// "does a step other than `self` touch buf within [b, e)?".
struct Touches {
    struct Iv { int32_t buf; int64_t b, e; size_t step; };
    std::vector<Iv> iv;
    std::vector<int64_t> maxlen;  // longest interval per buffer
    Touches(const XPhase& ph, int32_t n, bool reads, bool writes) : maxlen(size_t(n), 0) {
        for (size_t i = 0; i < ph.steps.size(); ++i) {
            const XStep& st = ph.steps[i];
            if (st.end <= st.begin) continue;
            if (reads) for (int32_t q : st.srcs) iv.push_back({q, st.begin, st.end, i});
            if (writes) for (int32_t q : st.dsts) iv.push_back({q, st.begin, st.end, i});
        }
        std::sort(iv.begin(), iv.end(), [](const Iv& x, const Iv& y) {
            return x.buf != y.buf ? x.buf < y.buf : x.b < y.b;
        });
        for (const Iv& x : iv) maxlen[size_t(x.buf)] = std::max(maxlen[size_t(x.buf)], x.e - x.b);
    }
    bool other(int32_t buf, int64_t b, int64_t e, size_t self) const {
        if (e <= b) return false;
        const int64_t from = b - maxlen[size_t(buf)];
        auto it = std::lower_bound(iv.begin(), iv.end(), std::make_pair(buf, from),
                                   [](const Iv& x, const std::pair<int32_t, int64_t>& k) {
                                       return x.buf != k.first ? x.buf < k.first : x.b < k.second;
                                   });
        for (; it != iv.end() && it->buf == buf && it->b < e; ++it)
            if (it->e > b && it->step != self) return true;
        return false;
    }
    bool any(int32_t buf, int64_t b, int64_t e) const {
        return other(buf, b, e, size_t(-1));
    }
};

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
static std::vector<XPhase> exec_phases(const Plan& p, bool fuse) {
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
static bool exec_phases_hazard_free(const std::vector<XPhase>& ph, int32_t n, std::string& why) {
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

// Group the steps of every executed phase by source count, choose the
// tiling and the cache mode of each launch.  Host only.
static void build_launches(const Plan& p, ExecState& ex) {
    const int64_t VEC = 16 / p.esize;
    ex.dev_of.assign(ex.phases.size(), {});
    for (size_t q = 0; q < ex.phases.size(); ++q) {
        const XPhase& xp = ex.phases[q];
        ex.dev_of[q].assign(xp.steps.size(), -1);
        std::unique_ptr<Touches> next_reads;
        if (q + 1 < ex.phases.size())
            next_reads.reset(new Touches(ex.phases[q + 1], p.n, true, false));
        std::vector<size_t> idx(xp.steps.size());
        for (size_t i = 0; i < idx.size(); ++i) idx[i] = i;
        // group by source count; inside a group, steps reading the same source
        // become neighbours (their repeated reads share cache)
        std::stable_sort(idx.begin(), idx.end(), [&](size_t a, size_t b) {
            const XStep& x = xp.steps[a];
            const XStep& y = xp.steps[b];
            if (x.srcs.size() != y.srcs.size()) return x.srcs.size() < y.srcs.size();
            if (x.srcs[0] != y.srcs[0]) return x.srcs[0] < y.srcs[0];
            return x.begin < y.begin;
        });
        size_t g0 = 0;
        while (g0 < idx.size()) {
            size_t g1 = g0;
            const int32_t k = int32_t(xp.steps[idx[g0]].srcs.size());
            while (g1 < idx.size() && int32_t(xp.steps[idx[g1]].srcs.size()) == k) ++g1;
            LaunchDesc L{};
            L.phase = xp.plan_phase;
            L.xphase = int32_t(q);
            L.kern_k = kernel_k(k);
            L.first = int64_t(ex.hsteps.size());
            L.count = int64_t(g1 - g0);
            int64_t maxspan = 0, bytes = 0, written = 0;
            int32_t maxdst = 0;
            std::vector<int64_t> spans;
            std::vector<std::tuple<int32_t, int64_t, int64_t>> ranges;
            bool next_reads_output = false;
            for (size_t g = g0; g < g1; ++g) {
                const XStep& x = xp.steps[idx[g]];
                DevStep d{};
                d.begin = x.begin;
                d.end = x.end;
                d.k = k;
                d.src_off = int32_t(ex.hidx.size());
                ex.hidx.insert(ex.hidx.end(), x.srcs.begin(), x.srcs.end());
                d.ndst = int32_t(x.dsts.size());
                d.dst_off = int32_t(ex.hidx.size());
                ex.hidx.insert(ex.hidx.end(), x.dsts.begin(), x.dsts.end());
                ex.dev_of[q][idx[g]] = int32_t(ex.hsteps.size());
                ex.hsteps.push_back(d);
                const int64_t len = x.end - x.begin;
                const int64_t span = len > 0 ? x.end - (x.begin & ~(VEC - 1)) : 0;
                spans.push_back(span);
                maxspan = std::max(maxspan, span);
                maxdst = std::max(maxdst, int32_t(x.dsts.size()));
                bytes += (k + int64_t(x.dsts.size())) * len * p.esize;
                written += int64_t(x.dsts.size()) * len * p.esize;
                if (len > 0) {
                    for (int32_t sidx : x.srcs) ranges.emplace_back(sidx, x.begin, x.end);
                    if (next_reads)
                        for (int32_t dd : x.dsts)
                            next_reads_output = next_reads_output || next_reads->any(dd, x.begin, x.end);
                }
            }
            L.bytes = bytes;
            L.max_dst = maxdst;
            L.rec_stride = (kRecHead + k + maxdst + 1) & ~int64_t(1);
            L.rec_off = ex.rec_words;
            ex.rec_of.resize(ex.hsteps.size(), -1);
            for (int64_t j = 0; j < L.count; ++j)
                ex.rec_of[size_t(L.first + j)] = L.rec_off + j * L.rec_stride;
            ex.rec_words += L.count * L.rec_stride;
            if (maxspan == 0) {  // nothing to move in this group
                g0 = g1;
                continue;
            }
            // wave tile: the measured best size for this source count,
            // halved while the launch has too few tiles to fill the chip
            const KCfg cfg = kcfg(L.kern_k);
            const int64_t tmin = int64_t(64) * cfg.U * VEC;
            int64_t te = int64_t(cfg.TE) * VEC;
            auto units_for = [&](int64_t t) {
                return L.count * ((maxspan + t - 1) / t);
            };
            while (te > tmin && units_for(te) < kMinUnits) te /= 2;
            while ((units_for(te) + cfg.WPB - 1) / cfg.WPB > kMaxBlocks) te *= 2;
            L.wpb = cfg.WPB;
            std::sort(ranges.begin(), ranges.end());
            const bool reuse = std::adjacent_find(ranges.begin(), ranges.end()) != ranges.end();
            L.cm = 0;
            if (bytes >= kNtBytes) {
                if (!reuse) L.cm |= 1;
                if (written > kKeepBytes || !next_reads_output) L.cm |= 2;
            }
            L.tile_elems = te;
            L.tiles_per_step = (maxspan + te - 1) / te;
            int64_t used = 0;
            for (int64_t sp : spans) used += (sp + te - 1) / te;
            if (used * 5 < L.count * L.tiles_per_step * 4) {
                // uneven steps: explicit tile table
                L.tile_off = int64_t(ex.htiles.size());
                for (int64_t j = 0; j < L.count; ++j) {
                    const int64_t nt = (spans[size_t(j)] + te - 1) / te;
                    for (int64_t t = 0; t < nt; ++t)
                        ex.htiles.push_back(make_int2(int(j), int(t)));
                }
                L.nunits = used;
            } else {
                L.tile_off = -1;
                L.nunits = L.count * L.tiles_per_step;
            }
            ex.launches.push_back(L);
            g0 = g1;
        }
    }
}

// The sliced launch of executed phases [p0, p1), if every boundary of their
// steps is 16-byte aligned.
static SliceDesc build_slice(const Plan& p, const ExecState& ex, int32_t p0, int32_t p1) {
    SliceDesc sd;
    const int64_t VEC = 16 / p.esize;
    sd.p0 = p0;
    sd.nphases = p1 - p0;
    for (int32_t q = p0; q < p1; ++q)
        for (const XStep& x : ex.phases[size_t(q)].steps)
            if (x.end > x.begin) {
                sd.cuts.push_back(x.begin);
                sd.cuts.push_back(x.end);
            }
    std::sort(sd.cuts.begin(), sd.cuts.end());
    sd.cuts.erase(std::unique(sd.cuts.begin(), sd.cuts.end()), sd.cuts.end());
    for (int64_t c : sd.cuts)
        if (c % VEC) {
            sd.why = "a step boundary is not 16-byte aligned";
            return sd;
        }
    if (sd.cuts.size() < 2) {
        sd.why = "nothing to move";
        return sd;
    }
    sd.nseg = int32_t(sd.cuts.size() - 1);
    if (int64_t(sd.nphases) * sd.nseg > (int64_t(1) << 24)) {
        sd.why = "too many phases times segments";
        return sd;
    }
    auto seg_of = [&](int64_t x) {  // segment starting at x
        return int32_t(std::lower_bound(sd.cuts.begin(), sd.cuts.end(), x) - sd.cuts.begin());
    };
    std::vector<std::vector<int32_t>> lists(size_t(sd.nphases) * size_t(sd.nseg));
    std::vector<char> used(size_t(sd.nseg), 0);
    for (int32_t q = p0; q < p1; ++q) {
        const XPhase& xp = ex.phases[size_t(q)];
        for (size_t i = 0; i < xp.steps.size(); ++i) {
            const XStep& x = xp.steps[i];
            if (x.end <= x.begin) continue;
            const int32_t di = ex.dev_of[size_t(q)][i];
            if (di < 0 || ex.rec_of[size_t(di)] < 0 || ex.rec_of[size_t(di)] > INT32_MAX) {
                sd.why = "step without a record";
                return sd;
            }
            for (int32_t sg = seg_of(x.begin); sg < seg_of(x.end); ++sg) {
                lists[size_t(q - p0) * size_t(sd.nseg) + size_t(sg)].push_back(
                    int32_t(ex.rec_of[size_t(di)]));
                used[size_t(sg)] = 1;
            }
            sd.bytes += (int64_t(x.srcs.size()) + int64_t(x.dsts.size())) * (x.end - x.begin) * p.esize;
            sd.max_k = std::max(sd.max_k, int32_t(x.srcs.size()));
            sd.max_dst = std::max(sd.max_dst, int32_t(x.dsts.size()));
            ++sd.nsteps;
        }
    }
    for (int32_t q = 0; q < sd.nphases; ++q) {
        size_t most = 0;
        for (int32_t sg = 0; sg < sd.nseg; ++sg)
            most = std::max(most, lists[size_t(q) * size_t(sd.nseg) + size_t(sg)].size());
        sd.chain += int64_t(most);
    }
    sd.sched_off.assign(lists.size() + 1, 0);
    for (size_t i = 0; i < lists.size(); ++i) {
        sd.sched_off[i + 1] = sd.sched_off[i] + int32_t(lists[i].size());
        sd.sched.insert(sd.sched.end(), lists[i].begin(), lists[i].end());
        if (sd.sched.size() > size_t(1) << 30) {
            sd.why = "schedule too large";
            return sd;
        }
    }
    sd.tile_elems = int64_t(64) * kSliceU * VEC;
    for (int32_t sg = 0; sg < sd.nseg; ++sg) {
        if (!used[size_t(sg)]) continue;
        const int64_t len = sd.cuts[size_t(sg) + 1] - sd.cuts[size_t(sg)];
        for (int64_t t = 0; t * sd.tile_elems < len; ++t) sd.tiles.push_back(make_int2(sg, int(t)));
    }
    sd.nunits = int64_t(sd.tiles.size());
    if ((sd.nunits + kSliceWPB - 1) / kSliceWPB > kMaxBlocks) {
        sd.why = "too many tiles";
        return sd;
    }
    sd.ok = sd.nunits > 0;
    if (!sd.ok) sd.why = "nothing to move";
    return sd;
}

// Per executed phase, what the choice of sliced runs needs: whether every
// step boundary is 16-byte aligned, the bytes written and moved, the most
// steps covering one element position, and the predicted phase-launch time.
struct PhaseCost {
    bool aligned = true;
    int64_t written = 0, read = 0, bytes = 0, cover = 0;
    int32_t kmax = 0, dmax = 0;
    double t_launch = 0.0;
};

static std::vector<PhaseCost> phase_costs(const Plan& p, const ExecState& ex) {
    const int64_t VEC = 16 / p.esize;
    std::vector<PhaseCost> pc(ex.phases.size());
    for (size_t q = 0; q < ex.phases.size(); ++q) {
        std::vector<std::pair<int64_t, int32_t>> ev;
        for (const XStep& x : ex.phases[q].steps) {
            if (x.end <= x.begin) continue;
            if (x.begin % VEC || x.end % VEC) pc[q].aligned = false;
            const int64_t len = x.end - x.begin;
            pc[q].written += int64_t(x.dsts.size()) * len * p.esize;
            pc[q].read += int64_t(x.srcs.size()) * len * p.esize;
            pc[q].kmax = std::max(pc[q].kmax, int32_t(x.srcs.size()));
            pc[q].dmax = std::max(pc[q].dmax, int32_t(x.dsts.size()));
            pc[q].bytes += (int64_t(x.srcs.size()) + int64_t(x.dsts.size())) * len * p.esize;
            ev.emplace_back(x.begin, 1);
            ev.emplace_back(x.end, -1);
        }
        std::sort(ev.begin(), ev.end());  // at equal positions ends (-1) first
        int64_t c = 0;
        for (const auto& e : ev) {
            c += e.second;
            pc[q].cover = std::max(pc[q].cover, c);
        }
    }
    for (const LaunchDesc& L : ex.launches)
        pc[size_t(L.xphase)].t_launch += kLaunchNs + double(L.bytes) / kBytesPerNs;
    return pc;
}

// Sliced runs for AR_OPT_SLICE = 2: phases [a, b), each aligned, writing at
// most kKeepBytes and moving at most kSliceMaxBytes, chosen to minimise the
// predicted time.  A run of one phase only pays off when it replaces
// several launches.
static std::vector<std::pair<int32_t, int32_t>> choose_runs(const Plan& p, const ExecState& ex,
                                                            const std::vector<PhaseCost>& pc) {
    const double per_src = p.dtype == AR_BF16 ? kStepNsPerSrcBF16 : kStepNsPerSrcF32;
    const double waves = std::max(1.0, double(p.N) * p.esize / (64.0 * kSliceU * 16.0));
    const double stretch = std::max(1.0, kMinSliceWaves / waves);
    const int32_t P = int32_t(pc.size());
    std::vector<int32_t> nl(size_t(P), 0);
    for (const LaunchDesc& L : ex.launches) ++nl[size_t(L.xphase)];
    std::vector<double> best(size_t(P) + 1, 0.0);
    std::vector<int32_t> from(size_t(P) + 1, -1);  // -1: phase launches for phase b - 1
    for (int32_t b = 1; b <= P; ++b) {
        best[size_t(b)] = best[size_t(b) - 1] + pc[size_t(b) - 1].t_launch;
        from[size_t(b)] = -1;
        double body = 0.0;
        for (int32_t a = b - 1; a >= 0; --a) {
            const PhaseCost& c = pc[size_t(a)];
            if (!c.aligned || c.written > kKeepBytes || c.bytes > kSliceMaxBytes) break;
            body += std::max({double(c.cover) * (kStepNs + per_src * c.kmax + kStepNsPerDst * c.dmax),
                              stretch * double(c.read) / kBytesPerNs,
                              double(c.written) / kBytesPerNs});
            if (b - a == 1 && nl[size_t(a)] < 2) continue;
            const double t = kLaunchNs + body;
            if (best[size_t(a)] + t < best[size_t(b)]) {
                best[size_t(b)] = best[size_t(a)] + t;
                from[size_t(b)] = a;
            }
        }
    }
    std::vector<std::pair<int32_t, int32_t>> runs;
    for (int32_t b = P; b > 0;) {
        if (from[size_t(b)] < 0) {
            --b;
        } else {
            runs.emplace_back(from[size_t(b)], b);
            b = from[size_t(b)];
        }
    }
    std::reverse(runs.begin(), runs.end());
    return runs;
}

static ExecState* exec_state(Plan& p) {
    if (!p.exec) {
        ExecState* ex = new ExecState();
        try {
            ex->phases = exec_phases(p, p.fuse != 0);
            build_launches(p, *ex);
            std::vector<std::pair<int32_t, int32_t>> runs;
            if (p.slice == 1 && !ex->phases.empty()) {
                runs.emplace_back(0, int32_t(ex->phases.size()));
            } else if (p.slice == 2) {
                runs = choose_runs(p, *ex, phase_costs(p, *ex));
            }
            std::vector<int32_t> slice_of(ex->phases.size(), -1);
            for (const auto& r : runs) {
                SliceDesc sd = build_slice(p, *ex, r.first, r.second);
                if (!sd.ok) continue;  // phase launches for these phases
                sd.cuts_base = ex->slices.empty() ? 0
                                                  : ex->slices.back().cuts_base +
                                                        int64_t(ex->slices.back().cuts.size());
                sd.soff_base = ex->slices.empty() ? 0
                                                  : ex->slices.back().soff_base +
                                                        int64_t(ex->slices.back().sched_off.size());
                sd.sched_base = ex->slices.empty() ? 0
                                                   : ex->slices.back().sched_base +
                                                         int64_t(ex->slices.back().sched.size());
                sd.tiles_base = ex->slices.empty() ? 0
                                                   : ex->slices.back().tiles_base +
                                                         int64_t(ex->slices.back().tiles.size());
                for (int32_t q = r.first; q < r.second; ++q)
                    slice_of[size_t(q)] = int32_t(ex->slices.size());
                ex->slices.push_back(std::move(sd));
            }
            int32_t last = -1;
            for (size_t li = 0; li < ex->launches.size(); ++li) {
                const int32_t sl = slice_of[size_t(ex->launches[li].xphase)];
                if (sl < 0) {
                    ex->stages.push_back({-1, int32_t(li)});
                } else if (sl != last) {
                    ex->stages.push_back({sl, -1});
                    last = sl;
                }
            }
        } catch (...) {
            delete ex;
            throw;
        }
        p.exec = ex;
    }
    return p.exec;
}

static void free_dev(DevState* d) {
    if (!d) return;
    int cur = -1;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(d->device);
    if (d->tiles) (void)hipFree(d->tiles);
    if (d->cuts) (void)hipFree(d->cuts);
    if (d->sched_off) (void)hipFree(d->sched_off);
    if (d->sched) (void)hipFree(d->sched);
    if (d->stiles) (void)hipFree(d->stiles);
    for (PtrEntry& e : d->cache) {
        if (e.done) {
            (void)hipEventSynchronize(e.done);
            (void)hipEventDestroy(e.done);
        }
        if (e.dev) (void)hipFree(e.dev);
        if (e.pinned) (void)hipHostFree(e.pinned);
    }
    if (cur >= 0) (void)hipSetDevice(cur);
    delete d;
}

void exec_release(Plan& p) {
    if (!p.exec) return;
    for (DevState* d : p.exec->dev) free_dev(d);
    delete p.exec;
    p.exec = nullptr;
}

template <class T>
static ar_status upload(T** dst, const std::vector<T>& src, const char* what) {
    if (src.empty()) return AR_OK;
    hipError_t e = hipMalloc(reinterpret_cast<void**>(dst), src.size() * sizeof(T));
    if (e != hipSuccess) {
        *dst = nullptr;
        (void)hipGetLastError();
        return fail(e == hipErrorOutOfMemory ? AR_ERR_OOM : AR_ERR_HIP,
                    hip_msg(what, e));
    }
    e = hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg(what, e));
    return AR_OK;
}

static ar_status device_state(Plan& p, ExecState& ex, DevState** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("hipGetDevice", e));
    if (dev < 0) return fail(AR_ERR_HIP, "no current device");
    if (size_t(dev) >= ex.dev.size()) ex.dev.resize(size_t(dev) + 1, nullptr);
    if (!ex.dev[size_t(dev)]) {
        DevState* d = new DevState();
        d->device = dev;
        ar_status s = upload(&d->tiles, ex.htiles, "tile table");
        if (s == AR_OK && !ex.slices.empty()) {
            std::vector<int64_t> cuts;
            std::vector<int32_t> soff, sched;
            std::vector<int2> tiles;
            for (const SliceDesc& sd : ex.slices) {
                cuts.insert(cuts.end(), sd.cuts.begin(), sd.cuts.end());
                soff.insert(soff.end(), sd.sched_off.begin(), sd.sched_off.end());
                sched.insert(sched.end(), sd.sched.begin(), sd.sched.end());
                tiles.insert(tiles.end(), sd.tiles.begin(), sd.tiles.end());
            }
            s = upload(&d->cuts, cuts, "segment table");
            if (s == AR_OK) s = upload(&d->sched_off, soff, "schedule offsets");
            if (s == AR_OK) s = upload(&d->sched, sched, "schedule");
            if (s == AR_OK) s = upload(&d->stiles, tiles, "slice tiles");
        }
        if (s != AR_OK) {
            free_dev(d);
            return s;
        }
        ex.dev[size_t(dev)] = d;
    }
    *out = ex.dev[size_t(dev)];
    (void)p;
    return AR_OK;
}

// Host-side checks of the buffer set: non-NULL and pairwise disjoint.
static ar_status check_buffers(const Plan& p, const std::vector<void*>& bufs) {
    const uint64_t bytes = uint64_t(p.N) * uint64_t(p.esize);
    std::vector<std::pair<uint64_t, int32_t>> a;
    a.reserve(bufs.size());
    for (size_t i = 0; i < bufs.size(); ++i) {
        if (!bufs[i])
            return fail(AR_ERR_INVALID_ARG, "buffer " + std::to_string(i) + " is NULL");
        a.emplace_back(reinterpret_cast<uint64_t>(bufs[i]), int32_t(i));
    }
    std::sort(a.begin(), a.end());
    for (size_t i = 1; i < a.size(); ++i)
        if (a[i].first < a[i - 1].first + bytes)
            return fail(AR_ERR_INVALID_ARG,
                        "buffers " + std::to_string(a[i - 1].second) + " and " +
                            std::to_string(a[i].second) + " overlap");
    return AR_OK;
}

// The step records for buffer set `bufs` on this device (see StepHead):
// from the per-plan cache, or built on the host and uploaded on `stream`.
static ar_status step_records(const Plan& p, const ExecState& ex, DevState& d,
                              const std::vector<void*>& bufs,
                              hipStream_t stream, PtrEntry** out) {
    ++d.clock;
    for (PtrEntry& e : d.cache)
        if (e.valid && e.key == bufs) {
            e.stamp = d.clock;
            *out = &e;
            return AR_OK;
        }
    ar_status s = check_buffers(p, bufs);
    if (s != AR_OK) return s;
    PtrEntry* v = &d.cache[0];
    for (PtrEntry& e : d.cache) {
        if (!e.valid) { v = &e; break; }
        if (e.stamp < v->stamp) v = &e;
    }
    const size_t nb = size_t(std::max<int64_t>(ex.rec_words, 1)) * sizeof(uint64_t);
    hipError_t e = hipSuccess;
    if (!v->dev) {
        e = hipMalloc(reinterpret_cast<void**>(&v->dev), nb);
        if (e != hipSuccess) {
            v->dev = nullptr;
            (void)hipGetLastError();
            return fail(e == hipErrorOutOfMemory ? AR_ERR_OOM : AR_ERR_HIP, hip_msg("step records", e));
        }
        e = hipHostMalloc(reinterpret_cast<void**>(&v->pinned), nb, hipHostMallocDefault);
        if (e != hipSuccess) {
            v->pinned = nullptr;
            (void)hipGetLastError();
            return fail(AR_ERR_OOM, hip_msg("step record staging", e));
        }
        e = hipEventCreateWithFlags(&v->done, hipEventDisableTiming);
        if (e != hipSuccess) {
            v->done = nullptr;
            return fail(AR_ERR_HIP, hip_msg("hipEventCreate", e));
        }
    } else {
        // the previous upload from the staging buffer must have finished
        e = hipEventSynchronize(v->done);
        if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("hipEventSynchronize", e));
    }
    v->valid = false;
    uint64_t* w = v->pinned;
    std::memset(w, 0, nb);
    for (size_t i = 0; i < ex.hsteps.size(); ++i) {
        const DevStep& st = ex.hsteps[i];
        uint64_t* r = w + ex.rec_of[i];
        StepHead h{st.begin, st.end, st.k, st.ndst, 0};
        std::memcpy(r, &h, sizeof(h));
        for (int32_t j = 0; j < st.k; ++j)
            r[kRecHead + j] = reinterpret_cast<uint64_t>(bufs[size_t(ex.hidx[size_t(st.src_off + j)])]);
        for (int32_t j = 0; j < st.ndst; ++j)
            r[kRecHead + st.k + j] =
                reinterpret_cast<uint64_t>(bufs[size_t(ex.hidx[size_t(st.dst_off + j)])]);
    }
    e = hipMemcpyAsync(v->dev, v->pinned, nb, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("step record upload", e));
    e = hipEventRecord(v->done, stream);
    if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("hipEventRecord", e));
    v->key = bufs;
    v->valid = true;
    v->stamp = d.clock;
    v->aligned = true;
    for (void* b : bufs)
        if (reinterpret_cast<uint64_t>(b) & 15) v->aligned = false;
    *out = v;
    return AR_OK;
}

template <int DT, int K>
static void launch_dk(bool vecok, int cm, int64_t blocks, hipStream_t st,
                      const uint64_t* recs, int64_t stride, const int2* tiles,
                      int64_t nunits, int64_t tps, int64_t te) {
    const dim3 grid(static_cast<uint32_t>(blocks)), block(64 * kcfg(K).WPB);
#define AR_LAUNCH(V, C)                                                                \
    hipLaunchKernelGGL((phase_kernel<DT, K, V, C>), grid, block, 0, st, recs, stride, \
                       tiles, nunits, tps, te)
    if (!vecok) AR_LAUNCH(false, 0);
    else if (cm == 0) AR_LAUNCH(true, 0);
    else if (cm == 1) AR_LAUNCH(true, 1);
    else if (cm == 2) AR_LAUNCH(true, 2);
    else AR_LAUNCH(true, 3);
#undef AR_LAUNCH
}

template <int DT>
static void launch_d(int K, bool vecok, int cm, int64_t blocks, hipStream_t st,
                     const uint64_t* recs, int64_t stride, const int2* tiles,
                     int64_t nunits, int64_t tps, int64_t te) {
    switch (K) {
        case 1: launch_dk<DT, 1>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te); break;
        case 2: launch_dk<DT, 2>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te); break;
        case 3: launch_dk<DT, 3>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te); break;
        case 4: launch_dk<DT, 4>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te); break;
        case 8: launch_dk<DT, 8>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te); break;
        case 16: launch_dk<DT, 16>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te); break;
        default: launch_dk<DT, 0>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te); break;
    }
}

}  // namespace arp

struct ar_timer {
    int64_t cap = 0;
    int64_t count = 0;
    std::vector<hipEvent_t> ev;  // 2 per record, created lazily
    std::vector<int32_t> launch;
};

using namespace arp;

static ar_status run(ar_plan* plan, const std::vector<void*>& bufs,
                     hipStream_t stream, ar_timer* timer) {
    try {
        if (plan->N == 0 || plan->num_phases() == 0) return AR_OK;
        ExecState* ex = exec_state(*plan);
        if (ex->launches.empty()) return AR_OK;
        DevState* d = nullptr;
        ar_status s = device_state(*plan, *ex, &d);
        if (s != AR_OK) return s;
        PtrEntry* pe = nullptr;
        s = step_records(*plan, *ex, *d, bufs, stream, &pe);
        if (s != AR_OK) return s;
        // sliced launches need 16-byte aligned buffers; otherwise every
        // phase runs as its phase launches
        const bool staged = pe->aligned;
        const int64_t nlaunch = staged ? int64_t(ex->stages.size()) : int64_t(ex->launches.size());
        if (timer && timer->count + nlaunch > timer->cap)
            return fail(AR_ERR_INVALID_ARG, "timer is full");
        auto mark = [&](int j) -> ar_status {  // event j (0 begin, 1 end) of this record
            if (!timer) return AR_OK;
            hipEvent_t& ev = timer->ev[size_t(2 * timer->count + j)];
            if (!ev) {
                hipError_t he = hipEventCreate(&ev);
                if (he != hipSuccess) {
                    ev = nullptr;
                    return fail(AR_ERR_HIP, hip_msg("hipEventCreate", he));
                }
            }
            hipError_t he = hipEventRecord(ev, stream);
            if (he != hipSuccess) return fail(AR_ERR_HIP, hip_msg("hipEventRecord", he));
            return AR_OK;
        };
        for (int64_t li = 0; li < nlaunch; ++li) {
            s = mark(0);
            if (s != AR_OK) return s;
            const Stage stg = staged ? ex->stages[size_t(li)] : Stage{-1, int32_t(li)};
            if (stg.slice >= 0) {
                const SliceDesc& sd = ex->slices[size_t(stg.slice)];
                const dim3 grid(static_cast<uint32_t>((sd.nunits + kSliceWPB - 1) / kSliceWPB));
                const dim3 block(64 * kSliceWPB);
#define AR_SLICED(DT)                                                                   \
    hipLaunchKernelGGL((sliced_kernel<DT>), grid, block, 0, stream, pe->dev,             \
                       d->sched_off + sd.soff_base, d->sched + sd.sched_base,           \
                       d->cuts + sd.cuts_base, d->stiles + sd.tiles_base, sd.nunits,    \
                       sd.nphases, sd.nseg, sd.tile_elems)
                switch (plan->dtype) {
                    case AR_F32: AR_SLICED(DT_F32); break;
                    case AR_I32: AR_SLICED(DT_I32); break;
                    default: AR_SLICED(DT_BF16); break;
                }
#undef AR_SLICED
            } else {
                const LaunchDesc& L = ex->launches[size_t(stg.launch)];
                const int64_t blocks = (L.nunits + L.wpb - 1) / L.wpb;
                const uint64_t* recs = pe->dev + L.rec_off;
                const int2* tiles = L.tile_off >= 0 ? d->tiles + L.tile_off : nullptr;
                switch (plan->dtype) {
                    case AR_F32:
                        launch_d<DT_F32>(L.kern_k, pe->aligned, L.cm, blocks, stream, recs,
                                         L.rec_stride, tiles, L.nunits, L.tiles_per_step,
                                         L.tile_elems);
                        break;
                    case AR_I32:
                        launch_d<DT_I32>(L.kern_k, pe->aligned, L.cm, blocks, stream, recs,
                                         L.rec_stride, tiles, L.nunits, L.tiles_per_step,
                                         L.tile_elems);
                        break;
                    default:
                        launch_d<DT_BF16>(L.kern_k, pe->aligned, L.cm, blocks, stream, recs,
                                          L.rec_stride, tiles, L.nunits, L.tiles_per_step,
                                          L.tile_elems);
                        break;
                }
            }
            hipError_t he = hipGetLastError();
            if (he != hipSuccess) return fail(AR_ERR_HIP, hip_msg("kernel launch", he));
            s = mark(1);
            if (s != AR_OK) return s;
            if (timer) timer->launch[size_t(timer->count++)] = int32_t(li);
        }
        return AR_OK;
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}

AR_EXPORT ar_status ar_plan_execute(ar_plan* plan, void* const* bufs, void* stream) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    if (!bufs) return fail(AR_ERR_INVALID_ARG, "bufs is NULL");
    return run(plan, std::vector<void*>(bufs, bufs + plan->n),
               static_cast<hipStream_t>(stream), nullptr);
}

AR_EXPORT ar_status ar_plan_execute_timed(ar_plan* plan, void* const* bufs, void* stream,
                                          ar_timer* timer) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    if (!bufs) return fail(AR_ERR_INVALID_ARG, "bufs is NULL");
    if (!timer) return fail(AR_ERR_INVALID_ARG, "timer is NULL");
    return run(plan, std::vector<void*>(bufs, bufs + plan->n),
               static_cast<hipStream_t>(stream), timer);
}

AR_EXPORT ar_status ar_plan_execute_strided(ar_plan* plan, void* base, int64_t stride_bytes,
                                            void* stream) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    if (!base) return fail(AR_ERR_INVALID_ARG, "base is NULL");
    if (stride_bytes < plan->N * plan->esize)
        return fail(AR_ERR_INVALID_ARG, "stride_bytes < N * element size");
    std::vector<void*> bufs(size_t(plan->n));
    for (int32_t i = 0; i < plan->n; ++i)
        bufs[size_t(i)] = static_cast<char*>(base) + int64_t(i) * stride_bytes;
    return run(plan, bufs, static_cast<hipStream_t>(stream), nullptr);
}

AR_EXPORT ar_status ar_timer_create(int64_t capacity, ar_timer** out) {
    clear_error();
    if (!out) return fail(AR_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (capacity < 1 || capacity > (int64_t(1) << 24))
        return fail(AR_ERR_INVALID_ARG, "capacity must be in [1, 2^24]");
    try {
        ar_timer* t = new ar_timer();
        t->cap = capacity;
        t->ev.assign(size_t(2 * capacity), nullptr);
        t->launch.assign(size_t(capacity), -1);
        *out = t;
        return AR_OK;
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    }
}

AR_EXPORT ar_status ar_timer_reset(ar_timer* timer) {
    clear_error();
    if (!timer) return fail(AR_ERR_INVALID_ARG, "timer is NULL");
    timer->count = 0;
    return AR_OK;
}

AR_EXPORT ar_status ar_timer_read(ar_timer* timer, int64_t cap, int64_t* count,
                                  int32_t* launch, float* ms) {
    clear_error();
    if (!timer || !count) return fail(AR_ERR_INVALID_ARG, "NULL argument");
    if (cap < 0) return fail(AR_ERR_INVALID_ARG, "cap < 0");
    const int64_t m = std::min(cap, timer->count);
    for (int64_t i = 0; i < m; ++i) {
        if (ms) {
            hipError_t e = hipEventSynchronize(timer->ev[size_t(2 * i + 1)]);
            if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("hipEventSynchronize", e));
            float t = 0.f;
            e = hipEventElapsedTime(&t, timer->ev[size_t(2 * i)], timer->ev[size_t(2 * i + 1)]);
            if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("hipEventElapsedTime", e));
            ms[i] = t;
        }
        if (launch) launch[i] = timer->launch[size_t(i)];
    }
    *count = m;
    return AR_OK;
}

AR_EXPORT ar_status ar_timer_destroy(ar_timer* timer) {
    clear_error();
    if (!timer) return AR_OK;
    for (hipEvent_t e : timer->ev)
        if (e) (void)hipEventDestroy(e);
    delete timer;
    return AR_OK;
}

// Host-side check of the executed phases and the launch tiling (no GPU):
// every executed phase is free of hazards, and walking every wave tile of
// every launch with the kernel's own index helpers covers each step exactly
// once, in bounds, with 16-byte aligned vector parts.  Declared in csrc/ar_debug.h (test hook, not part of the ABI).
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
            if (L.wpb != kcfg(L.kern_k).WPB) return bad("block size differs from the kernel's");
            if (L.tile_elems % (64 * VEC) != 0) return bad("tile not a multiple of a wave vector");
            const int2* tiles = L.tile_off >= 0 ? ex->htiles.data() + L.tile_off : nullptr;
            if (tiles && L.tile_off + L.nunits > int64_t(ex->htiles.size()))
                return bad("tile table overrun");
            for (int64_t j = 0; j < L.count; ++j) launched[size_t(L.first + j)] = 1;
            for (int64_t unit = 0; unit < blocks * L.wpb; ++unit) {
                if (unit >= L.nunits) continue;  // the kernel returns here
                int64_t s, t;
                unit_tile(unit, tiles, L.tiles_per_step, s, t);
                if (s < 0 || s >= L.count || t < 0) return bad("unit maps outside the launch");
                const DevStep& st = ex->hsteps[size_t(L.first + s)];
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
                cover[size_t(L.first + s)].push_back({sp.lo, sp.hi});
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
                if ((hi - lo) / VEC > 64 * kSliceU) return bad("slice tile too long");
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

AR_EXPORT ar_status ar_plan_set_option(ar_plan* plan, int32_t option, int64_t value) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    int32_t* field = nullptr;
    if (option == AR_OPT_FUSE) {
        if (value != 0 && value != 1) return fail(AR_ERR_INVALID_ARG, "AR_OPT_FUSE takes 0 or 1");
        field = &plan->fuse;
    } else if (option == AR_OPT_SLICE) {
        if (value < 0 || value > 2) return fail(AR_ERR_INVALID_ARG, "AR_OPT_SLICE takes 0, 1 or 2");
        field = &plan->slice;
    } else {
        return fail(AR_ERR_INVALID_ARG, "unknown option");
    }
    if (*field != int32_t(value)) {
        exec_release(*plan);
        *field = int32_t(value);
    }
    return AR_OK;
}

AR_EXPORT ar_status ar_plan_num_launches(const ar_plan* plan, int32_t* count) {
    clear_error();
    if (!plan || !count) return fail(AR_ERR_INVALID_ARG, "NULL argument");
    try {
        const ExecState* ex = exec_state(const_cast<ar_plan&>(*plan));
        *count = int32_t(ex->stages.size());
        return AR_OK;
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}

AR_EXPORT ar_status ar_plan_launch_info(const ar_plan* plan, int32_t i, int32_t* phase,
                                        int32_t* nsrc, int32_t* max_dst, int64_t* num_steps,
                                        int64_t* bytes) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    try {
        const ExecState* ex = exec_state(const_cast<ar_plan&>(*plan));
        if (i < 0 || i >= int32_t(ex->stages.size()))
            return fail(AR_ERR_INVALID_ARG, "launch index out of range");
        const Stage stg = ex->stages[size_t(i)];
        if (stg.slice >= 0) {
            const SliceDesc& sd = ex->slices[size_t(stg.slice)];
            if (phase) *phase = -1;
            if (nsrc) *nsrc = sd.max_k;
            if (max_dst) *max_dst = sd.max_dst;
            if (num_steps) *num_steps = sd.nsteps;
            if (bytes) *bytes = sd.bytes;
            return AR_OK;
        }
        const LaunchDesc& L = ex->launches[size_t(stg.launch)];
        if (phase) *phase = L.phase;
        if (nsrc) *nsrc = ex->hsteps[size_t(L.first)].k;
        if (max_dst) *max_dst = L.max_dst;
        if (num_steps) *num_steps = L.count;
        if (bytes) *bytes = L.bytes;
        return AR_OK;
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}
