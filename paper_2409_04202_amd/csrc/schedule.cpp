// Launch scheduling: executed phases become phase launches (steps grouped by
// source count, tiled, cache mode chosen) and sliced runs, plain or resident
// (their tables; the resident programs are built in programs.cpp), chosen by
// a cost model.  Host only.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <limits>
#include <map>
#include <memory>
#include <tuple>
#include <vector>

#include "exec_state.hpp"

namespace arp {

int kernel_k(int32_t k) {
    switch (k) {
        case 1: case 2: case 3: case 4: case 8: case 16: return k;
        default: return 0;
    }
}

// Tile table of a copy launch whose steps read some range more than once:
// the copies reading the same range are grouped, the range is cut into
// super-tiles of one workgroup's worth of tiles, and the super-tiles are
// dealt to the XCDs in turn, where one workgroup per copy runs each, one
// after the other: the repeated reads of a super-tile hit that XCD's L2
// instead of going to memory again, and each workgroup still writes one
// contiguous stretch (dealing them by position instead, as xcd_of does,
// measured slower: the tree (8, 8)'s last AllGather 152 -> 179 us).  Workgroups are dispatched to the kNumXCDs XCDs
// round-robin by workgroup id, so workgroup b runs on XCD b % kNumXCDs; the
// table gives each XCD the same number of workgroups, padding with entries
// (-1, 0) that the kernel skips.  Used for copies of at most kXcdMaxTiles tiles: the repeated reads
// of longer copies come far enough apart for the last-level cache, shared by
// all XCDs, to serve them, and their writes streamed better without the
// grouping (measured).  Steps are idx[g0..g1) of executed phase xp, in
// launch order.
static bool xcd_tiles(const XPhase& xp, const std::vector<size_t>& idx, size_t g0, size_t g1,
                      int64_t te, int64_t VEC, LaunchDesc& L, ExecState& ex) {
    std::map<std::tuple<int32_t, int64_t, int64_t>, std::vector<int32_t>> groups;
    for (size_t g = g0; g < g1; ++g) {
        const XStep& x = xp.steps[idx[g]];
        if (x.end > x.begin)
            groups[std::make_tuple(x.srcs[0], x.begin, x.end)].push_back(int32_t(g - g0));
    }
    const int64_t wpb = L.wpb;
    std::vector<std::vector<int2>> seq(static_cast<size_t>(kNumXCDs));
    size_t next_xcd = 0;
    for (const auto& gr : groups) {
        const XStep& x = xp.steps[idx[g0 + size_t(gr.second[0])]];
        const int64_t nt = (x.end - (x.begin & ~(VEC - 1)) + te - 1) / te;
        for (int64_t t0 = 0; t0 < nt; t0 += wpb) {
            std::vector<int2>& q = seq[next_xcd];
            next_xcd = (next_xcd + 1) % size_t(kNumXCDs);
            for (int32_t j : gr.second)
                for (int64_t t = t0; t < t0 + wpb; ++t)
                    q.push_back(t < nt ? make_int2(j, int(t)) : make_int2(-1, 0));
        }
    }
    size_t len = 0;
    for (const auto& q : seq) len = std::max(len, q.size());
    const int64_t nunits = int64_t(len) * kNumXCDs;
    if ((nunits + wpb - 1) / wpb > kMaxBlocks) return false;
    L.tile_off = int64_t(ex.htiles.size());
    for (size_t q0 = 0; q0 < len; q0 += size_t(wpb))  // block q0 / wpb of each XCD
        for (size_t x = 0; x < size_t(kNumXCDs); ++x)
            for (size_t u = q0; u < q0 + size_t(wpb); ++u)
                ex.htiles.push_back(u < seq[x].size() ? seq[x][u] : make_int2(-1, 0));
    L.nunits = nunits;
    return true;
}

// Affinity table: each tile goes to the XCD xcd_of its first element.
// Workgroups are dispatched to the XCDs round-robin by workgroup id, so
// workgroup b runs on XCD b % kNumXCDs: the table gives each XCD's
// workgroups its tiles in launch order, padding with entries (-1, 0) that
// the kernel skips.  A split launch (dsplit > 1) has one tile per
// workgroup, others wpb.  Steps are idx[g0..g1) of executed phase xp, in
// launch order, spans[j] the element span of step g0 + j.
static void affinity_tiles(const XPhase& xp, const std::vector<size_t>& idx, size_t g0,
                           size_t g1, const std::vector<int64_t>& spans, int64_t te,
                           int64_t VEC, int64_t N, LaunchDesc& L, ExecState& ex) {
    std::vector<std::vector<int2>> seq(static_cast<size_t>(kNumXCDs));
    for (size_t j = 0; j < g1 - g0; ++j) {
        const XStep& x = xp.steps[idx[g0 + j]];
        const int64_t abase = x.begin & ~(VEC - 1);
        for (int64_t t = 0; t * te < spans[j]; ++t) {
            const int64_t lo = std::max(abase + t * te, x.begin);
            seq[size_t(xcd_of(lo, N))].push_back(make_int2(int(j), int(t)));
        }
    }
    const size_t per_wg = L.dsplit > 1 ? 1 : size_t(L.wpb);
    size_t len = 0;
    for (const auto& q : seq) len = std::max(len, (q.size() + per_wg - 1) / per_wg * per_wg);
    L.tile_off = int64_t(ex.htiles.size());
    for (size_t q0 = 0; q0 < len; q0 += per_wg)
        for (size_t x = 0; x < size_t(kNumXCDs); ++x)
            for (size_t u = q0; u < q0 + per_wg; ++u)
                ex.htiles.push_back(u < seq[x].size() ? seq[x][u] : make_int2(-1, 0));
    L.nunits = int64_t(len * size_t(kNumXCDs)) * L.dsplit;
    L.affinity = 1;
}

// Group the steps of every executed phase by source count, choose the
// tiling and the cache mode of each launch.  Host only.
static void build_launches(const Plan& p, ExecState& ex) {
    const int64_t VEC = 16 / p.esize;
    ex.dev_of.assign(ex.phases.size(), {});
    // the previous executed phase: every launch kept its stores cached, and
    // the bytes it wrote
    bool prev_kept = false;
    int64_t prev_written = 0;
    for (size_t q = 0; q < ex.phases.size(); ++q) {
        const XPhase& xp = ex.phases[q];
        ex.dev_of[q].assign(xp.steps.size(), -1);
        bool all_kept = true;
        int64_t phase_written = 0;
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
                // destinations that are not sources of the step first
                d.ndst = int32_t(x.dsts.size());
                d.dst_off = int32_t(ex.hidx.size());
                for (int pass = 0; pass < 2; ++pass)
                    for (int32_t dd : x.dsts) {
                        const bool src =
                            std::find(x.srcs.begin(), x.srcs.end(), dd) != x.srcs.end();
                        if (src == (pass == 1)) ex.hidx.push_back(dd);
                    }
                d.nfree = d.ndst;
                for (int32_t dd : x.dsts)
                    if (std::find(x.srcs.begin(), x.srcs.end(), dd) != x.srcs.end()) --d.nfree;
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
            L.rt_group = L.kern_k == 0 && bytes < kRtGroupMaxBytes ? kRtGroup : 1;
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
            const int64_t min_units = k >= 2 ? kMinUnitsReduce : kMinUnits;
            std::sort(ranges.begin(), ranges.end());
            const bool reuse = std::adjacent_find(ranges.begin(), ranges.end()) != ranges.end();
            while (te > tmin && units_for(te) < min_units) te /= 2;
            // still too few tiles: below the kernel's full pass, down to one
            // vector per lane (copies reading a range several times keep
            // their XCD tables' tile size; many-destination steps split)
            if (bytes >= kFineTileMinBytes && !(k == 1 && reuse) && maxdst < kSplitMinDst)
                while (te > 64 * VEC && units_for(te) < kMinUnits) te /= 2;
            while ((units_for(te) + cfg.WPB - 1) / cfg.WPB > kMaxBlocks) te *= 2;
            L.wpb = cfg.WPB;
            L.cm = 0;
            if (bytes >= kNtBytes) {
                // a fold reading what the previous phase left in the cache
                // loads through it
                const bool warm = k >= 2 && prev_kept && prev_written <= kWarmBytes;
                if (!reuse && !warm) L.cm |= 1;
                const int64_t keep = k >= 2 ? kKeepBytesFold : kKeepBytes;
                if (written > keep || !next_reads_output) L.cm |= 2;
            }
            L.wide = (L.kern_k == 2 && L.cm == 3 && bytes >= kWideBytes &&
                      maxdst < kSplitMinDst && te == int64_t(64) * kWideU * VEC &&
                      te == int64_t(cfg.TE) * VEC) ||
                     (L.kern_k == 8 && p.esize == 4 && (L.cm & 1) && bytes >= kWideBytes &&
                      maxdst < kSplitMinDst && te == int64_t(64) * kWideU8 * VEC &&
                      te == int64_t(cfg.TE) * VEC);
            all_kept = all_kept && !(L.cm & 2);
            phase_written += written;
            L.tile_elems = te;
            L.tiles_per_step = (maxspan + te - 1) / te;
            int64_t used = 0;
            for (int64_t sp : spans) used += (sp + te - 1) / te;
            // few tiles storing to many destinations: a workgroup per tile
            L.dsplit = 1;
            if (maxdst >= kSplitMinDst && used < kMinUnits &&
                (bytes < kNtBytes || maxdst >= kSplitWideDst * k))
                L.dsplit = L.wpb = kSplitWaves;
            // copies reading the same range run next to each other (or on one
            // XCD, below): their repeated reads hit the cache
            L.hbm = bytes;
            if (k == 1 && reuse) {
                L.hbm = written;
                for (size_t r = 0; r < ranges.size(); ++r)
                    if (r == 0 || ranges[r] != ranges[r - 1])
                        L.hbm += (std::get<2>(ranges[r]) - std::get<1>(ranges[r])) * p.esize;
            }
            const bool xcd_copy = k == 1 && reuse && L.tiles_per_step <= kXcdMaxTiles;
            const bool affinity =
                L.dsplit > 1 ||
                (!xcd_copy && (bytes <= kAffinityMaxBytes ||
                               (bytes >= kAffinityBigBytes && !reuse && k <= 2)));
            if (affinity) {
                affinity_tiles(xp, idx, g0, g1, spans, te, VEC, p.N, L, ex);
            } else if (xcd_copy &&
                xcd_tiles(xp, idx, g0, g1, te, VEC, L, ex)) {
                // copies reading the same range run on one XCD (tile table)
            } else if (used * 5 < L.count * L.tiles_per_step * 4) {
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
        prev_kept = all_kept;
        prev_written = phase_written;
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
    bool short_many = false;  // a step to >= kSplitMinDst buffers, short
    uint64_t touched = 0;  // buffers the phase touches (n <= kResMaxN)
    double t_launch = 0.0;
};

// Bytes per ns of the cost model: the cached rate when the plan's whole
// footprint fits the last-level cache.
static double byte_rate(const Plan& p) {
    return int64_t(p.n) * p.N * p.esize <= kCacheBytes ? kCachedBytesPerNs : kBytesPerNs;
}

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
            pc[q].short_many = pc[q].short_many ||
                               (int32_t(x.dsts.size()) >= kSplitMinDst &&
                                len * p.esize < kSlicedManyDstMinBytes);
            pc[q].bytes += (int64_t(x.srcs.size()) + int64_t(x.dsts.size())) * len * p.esize;
            if (p.n <= kResMaxN) {
                for (int32_t b : x.srcs) pc[q].touched |= uint64_t(1) << b;
                for (int32_t b : x.dsts) pc[q].touched |= uint64_t(1) << b;
            }
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
    const double bpn = byte_rate(p);
    for (const LaunchDesc& L : ex.launches) {
        // dependent rounds of loads: a runtime-source-count fold loads its
        // sources rt_group at a time
        const int64_t k = ex.hsteps[size_t(L.first)].k;
        const double rounds = L.kern_k == 0 ? double((k + L.rt_group - 1) / L.rt_group) : 1.0;
        pc[size_t(L.xphase)].t_launch +=
            kPhaseLaunchNs + std::max(kKernelMinNs * rounds, double(L.hbm) / bpn);
    }
    return pc;
}

// Sliced runs for AR_OPT_SLICE = 2: phases [a, b), each aligned, chosen to
// minimise the predicted time, each in its plain form (phases writing at most
// kKeepBytes and moving at most kSliceMaxBytes) or (AR_OPT_RESIDENT,
// n <= kResMaxN) its resident form, whichever is predicted faster.  A run of
// one phase that replaces a single launch must be predicted kSingleRunGain
// of that launch's time or less.
struct Run {
    int32_t a, b;
    bool resident;
};

static std::vector<Run> choose_runs(const Plan& p, const ExecState& ex,
                                    const std::vector<PhaseCost>& pc, double* t_total) {
    const double per_src = p.dtype == AR_BF16 ? kStepNsPerSrcBF16 : kStepNsPerSrcF32;
    const double bpn = byte_rate(p);
    const double waves = std::max(1.0, double(p.N) * p.esize / (64.0 * kSliceU * 16.0));
    const double stretch = std::max(1.0, kMinSliceWaves / waves);
    const bool res_ok = p.resident != 0 && p.n <= kResMaxN;
    // resident tiles (one vector per lane), their workgroup size, and how
    // many run at once
    const double tiles = std::max(1.0, double(p.N) * p.esize / (64.0 * 16.0));
    const int32_t W = res_waves(p.n, int64_t(tiles));
    const int64_t per_cu = std::max<int64_t>(
        1, std::min<int64_t>(W == 4 ? 8 : kResWavesPerCU, kLdsBytesPerCU / (int64_t(p.n) * 1024)));
    // workgroups sharing a compute unit when the tiles are spread evenly
    const double sharing = std::min(double(per_cu), std::ceil(tiles / double(kNumCUs)));
    const double rounds = std::ceil(tiles / double(kNumCUs * per_cu)) *
                          (1.0 + kResShare * (sharing - 1.0));
    const int32_t P = int32_t(pc.size());
    std::vector<int32_t> nl(size_t(P), 0);
    for (const LaunchDesc& L : ex.launches) ++nl[size_t(L.xphase)];
    std::vector<double> best(size_t(P) + 1, 0.0);
    std::vector<int32_t> from(size_t(P) + 1, -1);  // -1: phase launches for phase b - 1
    std::vector<char> res_of(size_t(P) + 1, 0);
    for (int32_t b = 1; b <= P; ++b) {
        best[size_t(b)] = best[size_t(b) - 1] + pc[size_t(b) - 1].t_launch;
        from[size_t(b)] = -1;
        double body = 0.0, chain = 0.0;
        uint64_t touched = 0;
        bool next_link = false;
        // a plain sliced run hands data between its phases through the
        // cache, so its phases must be small; a resident run keeps them in
        // LDS and takes phases of any size
        bool plain_ok = true;
        for (int32_t a = b - 1; a >= 0; --a) {
            const PhaseCost& c = pc[size_t(a)];
            if (!c.aligned) break;
            plain_ok = plain_ok && c.written <= kKeepBytes && c.bytes <= kSliceMaxBytes &&
                       !(p.n > kResMaxN && c.short_many);
            if (!plain_ok && !res_ok) break;
            body += std::max({double(c.cover) * (kStepNs + per_src * c.kmax + kStepNsPerDst * c.dmax),
                              stretch * double(c.read) / bpn,
                              double(c.written) / bpn});
            // a run is priced from its last phase down: phase a chains into
            // phase a + 1 when both have one 2-source step per position
            const bool link = c.cover == 1 && c.kmax == 2 && c.dmax == 1;
            // the run's last phase stores its further destinations through
            // the alias table, at no step cost
            const int32_t d = a == b - 1 ? 1 : c.dmax;
            chain += link && next_link ? kResChainNs
                     : double(c.cover) *
                           (c.kmax <= 2 && d == 1
                                ? kResFastNs
                                : kResStepNs + kResStepNsPerSrc * c.kmax + kResStepNsPerDst * d);
            next_link = link;
            touched |= c.touched;
            // a run of one phase that replaces a single launch: only when
            // predicted far cheaper (the estimate for one phase is optimistic)
            const bool single = b - a == 1 && nl[size_t(a)] < 2;
            double t = plain_ok ? kLaunchNs + body : std::numeric_limits<double>::infinity();
            bool res = false;
            if (res_ok) {
                const double rows = 2.0 * double(__builtin_popcountll(touched));
                const double t_waves = rounds * (kResRowNs / W * rows + chain);
                const double t_bytes = rows * double(p.N) * p.esize / bpn;
                const double t_res = kLaunchNs + (a > 0 ? kResAfterLaunchNs : 0.0) +
                                     std::max(t_waves, t_bytes) +
                                     kResOverlap * std::min(t_waves, t_bytes);
                if (t_res < t) {
                    t = t_res;
                    res = true;
                }
            }
            if (single && !(t < kSingleRunGain * pc[size_t(a)].t_launch)) continue;
            if (best[size_t(a)] + t < best[size_t(b)]) {
                best[size_t(b)] = best[size_t(a)] + t;
                from[size_t(b)] = a;
                res_of[size_t(b)] = res;
            }
        }
    }
    *t_total = best[size_t(P)];
    std::vector<Run> runs;
    for (int32_t b = P; b > 0;) {
        if (from[size_t(b)] < 0) {
            --b;
        } else {
            runs.push_back({from[size_t(b)], b, res_of[size_t(b)] != 0});
            b = from[size_t(b)];
        }
    }
    std::reverse(runs.begin(), runs.end());
    return runs;
}

// Predicted time of a streamed launch (see kStreamWordNs).
static double stream_time(const Plan& p, const SliceDesc& sd) {
    const int64_t lds = int64_t(sd.slots) * 1024 + int64_t(p.n) * 8 + int64_t(sd.max_nw) * 4;
    const int64_t per_cu = std::max<int64_t>(1, kLdsBytesPerCU / lds);
    const double rounds = std::ceil(double(sd.nunits) / double(kNumCUs * per_cu));
    return kLaunchNs + rounds * double(sd.max_nw) * kStreamWordNs;
}

static std::atomic<uint64_t> g_exec_serial{0};

ExecState* exec_state(Plan& p) {
    if (!p.exec) {
        ExecState* ex = new ExecState();
        ex->serial = ++g_exec_serial;
        try {
            ex->phases = exec_phases(p, p.fuse != 0);
            build_launches(p, *ex);
            std::vector<Run> runs;
            const int32_t P = int32_t(ex->phases.size());
            SliceDesc streamed;  // the whole plan streamed, when chosen below
            bool have_streamed = false;
            if (p.slice == 1 && P > 0) {
                runs.push_back({0, P, p.resident != 0});
            } else if (p.slice == 2) {
                double t_runs = 0.0;
                runs = choose_runs(p, *ex, phase_costs(p, *ex), &t_runs);
                if (p.resident != 0 && p.n > kResMaxN && P > 0) {
                    SliceDesc sd = build_slice(p, *ex, 0, P);
                    if (sd.ok) {
                        build_resident(p, *ex, sd);
                        if (sd.streamed && stream_time(p, sd) < kStreamGain * t_runs) {
                            runs.assign(1, Run{0, P, true});
                            streamed = std::move(sd);
                            have_streamed = true;
                        }
                    }
                }
            }
            std::vector<int32_t> slice_of(ex->phases.size(), -1);
            for (const Run& r : runs) {
                SliceDesc sd = have_streamed ? std::move(streamed) : build_slice(p, *ex, r.a, r.b);
                if (!sd.ok) continue;  // phase launches for these phases
                if (r.resident && !have_streamed) build_resident(p, *ex, sd);
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
                sd.runit_base = ex->slices.empty() ? 0
                                                   : ex->slices.back().runit_base +
                                                         int64_t(ex->slices.back().runits.size());
                sd.prog_base = ex->slices.empty() ? 0
                                                  : ex->slices.back().prog_base +
                                                        int64_t(ex->slices.back().prog.size());
                for (int32_t q = r.a; q < r.b; ++q)
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

}  // namespace arp
