// Launch scheduling: executed phases become phase launches (steps grouped by
// source count, tiled, cache mode chosen) and sliced runs, plain or resident
// (their tables, and the resident programs), chosen by a cost model.  Host
// only.
#include <algorithm>
#include <cmath>
#include <functional>
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
// super-tiles of one workgroup's worth of tiles, and each super-tile is dealt
// to one XCD, where one workgroup per copy runs it, one after the other: the
// repeated reads of a super-tile hit that XCD's L2 instead of going to
// memory again, and each workgroup still writes one contiguous stretch.
// Workgroups are dispatched to the kNumXCDs XCDs round-robin by workgroup
// id, so workgroup b runs on XCD b % kNumXCDs; the table gives each XCD the
// same number of workgroups, padding with entries (-1, 0) that the kernel
// skips.  Used for copies of at most kXcdMaxTiles tiles: the repeated reads
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
            // copies reading the same range run next to each other (or on one
            // XCD, below): their repeated reads hit the cache
            L.hbm = bytes;
            if (k == 1 && reuse) {
                L.hbm = written;
                for (size_t r = 0; r < ranges.size(); ++r)
                    if (r == 0 || ranges[r] != ranges[r - 1])
                        L.hbm += (std::get<2>(ranges[r]) - std::get<1>(ranges[r])) * p.esize;
            }
            if (k == 1 && reuse && L.tiles_per_step <= kXcdMaxTiles &&
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

// Wavefronts per resident workgroup: four issue a tile's row loads and
// stores in parallel, which pays when LDS already limits a compute unit to
// at most eight tiles (32 waves) or when there are too few tiles to fill the
// chip; otherwise one wave per tile lets a unit hold more tiles.
static int32_t res_waves(int32_t n, int64_t units) {
    const int64_t by_lds = kLdsBytesPerCU / (int64_t(n) * 1024);
    return by_lds <= 8 || units <= 4 * kNumCUs ? 4 : 1;
}

// Resident records of the steps covering one segment, in phase order
// (encoding: resident_kernel).  Two-source steps that each fold the previous
// one's result, whose intermediate results nothing reads later (the next
// touch of such a row after the step that consumes it overwrites it), become
// one chain record that keeps the running result in registers and writes
// only the last one.
static void encode_segment(const std::vector<const XStep*>& st, std::vector<uint32_t>& w,
                           std::vector<uint8_t>& alias) {
    alias.assign(64, 0xFF);
    const size_t L = st.size();
    std::vector<uint64_t> rd(L, 0), wr(L, 0);
    for (size_t j = 0; j < L; ++j) {
        for (int32_t b : st[j]->srcs) rd[j] |= uint64_t(1) << b;
        for (int32_t b : st[j]->dsts) wr[j] |= uint64_t(1) << b;
    }
    // next[j * 64 + r]: the first record after j touching row r, or -1
    std::vector<int32_t> next(L * 64, -1);
    for (size_t j = L; j-- > 0;) {
        if (j + 1 < L) {
            std::copy(next.begin() + (j + 1) * 64, next.begin() + (j + 2) * 64, next.begin() + j * 64);
            for (int r = 0; r < 64; ++r)
                if ((rd[j + 1] | wr[j + 1]) >> r & 1) next[j * 64 + r] = int32_t(j + 1);
        }
    }
    auto add2 = [&](size_t j) { return st[j]->srcs.size() == 2 && st[j]->dsts.size() == 1; };
    // can record j's result stay in registers for record j + 1 only?
    auto chained = [&](size_t j) {
        if (j + 1 >= L || !add2(j) || !add2(j + 1)) return false;
        const int32_t d = st[j]->dsts[0];
        const XStep& x = *st[j + 1];
        if ((x.srcs[0] == d) == (x.srcs[1] == d)) return false;  // exactly one operand
        if (wr[j + 1] >> d & 1) return true;                      // overwritten at once
        const int32_t t = next[(j + 1) * 64 + size_t(d)];
        return t >= 0 && (wr[size_t(t)] >> d & 1) && !(rd[size_t(t)] >> d & 1);
    };
    auto put = [&](const std::vector<uint32_t>& rec) {
        if (w.size() % 64 + rec.size() > 64) w.resize((w.size() + 63) / 64 * 64, 0u);
        w.insert(w.end(), rec.begin(), rec.end());
    };
    std::vector<uint32_t> rec;
    for (size_t j = 0; j < L;) {
        if (chained(j)) {
            size_t j1 = j + 1;  // the chain is records j..j1
            while (j1 - j + 1 < 64 && chained(j1)) ++j1;
            const size_t m = j1 - j + 1;
            std::vector<int32_t> ys{st[j]->srcs[1]};
            for (size_t i = j + 1; i <= j1; ++i) {
                const int32_t prev = st[i - 1]->dsts[0];
                ys.push_back(st[i]->srcs[0] == prev ? st[i]->srcs[1] : st[i]->srcs[0]);
            }
            rec.assign(1 + (m + 3) / 4, 0u);
            rec[0] = kResChain | uint32_t(m) << 8 | uint32_t(st[j]->srcs[0]) << 16 |
                     uint32_t(st[j1]->dsts[0]) << 24;
            for (size_t i = 0; i < m; ++i) rec[1 + i / 4] |= uint32_t(ys[i]) << (8 * (i % 4));
            put(rec);
            j = j1 + 1;
            continue;
        }
        const XStep& x = *st[j];
        const size_t k = x.srcs.size();
        // the fold, add or copy into the first destination
        if (k == 2) {
            rec.assign(1, kResAdd2 | uint32_t(x.srcs[0]) << 8 | uint32_t(x.srcs[1]) << 16 |
                              uint32_t(x.dsts[0]) << 24);
        } else if (k == 1) {
            rec.assign(1, kResCopy | uint32_t(x.srcs[0]) << 8 | uint32_t(x.srcs[0]) << 16 |
                              uint32_t(x.dsts[0]) << 24);
        } else {
            rec.assign(1 + (k + 3) / 4, 0u);
            rec[0] = kResFold | uint32_t(k) << 8 | uint32_t(x.dsts[0]) << 16;
            for (size_t i = 0; i < k; ++i) rec[1 + i / 4] |= uint32_t(x.srcs[i]) << (8 * (i % 4));
        }
        put(rec);
        // then the same value into the other destinations: when nothing
        // touches them afterwards and nothing writes the first one, the
        // store pass takes their values from the first one's row (alias);
        // otherwise a store record, its list padded to a multiple of four by
        // repeating its last row
        bool aliased = x.dsts.size() > 1;
        for (size_t i = 1; i < x.dsts.size() && aliased; ++i)
            aliased = next[j * 64 + size_t(x.dsts[i])] < 0;
        for (size_t i = j + 1; i < L && aliased; ++i) aliased = !(wr[i] >> x.dsts[0] & 1);
        if (aliased) {
            for (size_t i = 1; i < x.dsts.size(); ++i) alias[size_t(x.dsts[i])] = uint8_t(x.dsts[0]);
        } else if (x.dsts.size() > 1) {
            std::vector<int32_t> ds(x.dsts.begin() + 1, x.dsts.end());
            while (ds.size() % 4) ds.push_back(ds.back());
            rec.assign(1 + ds.size() / 4, 0u);
            rec[0] = kResStore | uint32_t(ds.size()) << 8;
            for (size_t i = 0; i < ds.size(); ++i) rec[1 + i / 4] |= uint32_t(ds[i]) << (8 * (i % 4));
            put(rec);
        }
        ++j;
    }
}

// Streamed program of one segment (stream_kernel, encoding in resident.hpp):
// the steps st (phase order) of a run over n buffers become values (a
// buffer's row as the run finds it, or a step's fold of k >= 2 values; a
// copy names its source's value), the values that some buffer ends with are
// computed depth first (each fold after its inputs, in source order) and
// stored into those buffers at once, each value holds a slot from its load or
// fold to its last use, and the rows are loaded kStreamAhead rows ahead of
// their first use, with a wait for a load before its value is read (until at
// most as many memory operations are outstanding as loads followed it).  A store
// into a buffer whose row the segment still has to load waits until the end.
// Fills w (64-word chunks) and the slots, loads and stores it uses; false when
// a fold has more than 252 sources or the slots run out.
constexpr int32_t kStreamAhead = 48;
// waves of a streamed workgroup (the kernel takes 1 or 4; one wave owning
// the whole tile measured the same as four owning a quarter each)
constexpr int32_t kStreamWaves = 4;
constexpr size_t kStreamReserve = 2;  // slots kept for fold results

static bool encode_stream(const std::vector<const XStep*>& st, int32_t n,
                          std::vector<uint32_t>& w, int32_t& nslots, int64_t& nload,
                          int64_t& nstore) {
    struct Val {
        int32_t leaf;                // buffer whose row it is, or -1 (a fold)
        std::vector<int32_t> in;     // a fold's inputs in source order
    };
    std::vector<Val> vals;
    std::vector<int32_t> cur(size_t(n), -1), leaf_of(size_t(n), -1);
    std::vector<char> written(size_t(n), 0);
    for (const XStep* x : st) {
        std::vector<int32_t> in;
        for (int32_t b : x->srcs) {
            if (cur[size_t(b)] < 0) {  // first touched by a read: its row
                leaf_of[size_t(b)] = cur[size_t(b)] = int32_t(vals.size());
                vals.push_back({b, {}});
            }
            in.push_back(cur[size_t(b)]);
        }
        int32_t out = in[0];
        if (in.size() > 252) return false;  // a fold record fits a 64-word chunk
        if (in.size() > 1) {
            out = int32_t(vals.size());
            vals.push_back({-1, std::move(in)});
        }
        // the phases are hazard-free: no later step of this phase reads a
        // destination, so updating at once keeps phase-start reads
        for (int32_t d : x->dsts) {
            cur[size_t(d)] = out;
            written[size_t(d)] = 1;
        }
    }
    const size_t V = vals.size();
    std::vector<std::vector<int32_t>> puts(V);
    for (int32_t b = 0; b < n; ++b)
        if (written[size_t(b)] && cur[size_t(b)] != leaf_of[size_t(b)])
            puts[size_t(cur[size_t(b)])].push_back(b);
    // computing order: depth first from each stored value; then the leaves
    // in the order of their first use
    std::vector<char> seen(V, 0);
    std::vector<int32_t> events;  // fold v: v; store of v: -1 - v
    std::vector<int32_t> uses(V, 0);
    std::function<void(int32_t)> visit = [&](int32_t v) {
        if (seen[size_t(v)]) return;
        seen[size_t(v)] = 1;
        for (int32_t i : vals[size_t(v)].in) {
            visit(i);
            ++uses[size_t(i)];
        }
        if (vals[size_t(v)].leaf < 0) events.push_back(v);
    };
    for (size_t v = 0; v < V; ++v)
        if (!puts[v].empty()) {
            visit(int32_t(v));
            ++uses[v];
            events.push_back(-1 - int32_t(v));
        }
    std::vector<int32_t> q;  // leaves by first use
    std::vector<char> queued(V, 0);
    for (int32_t e : events) {
        const int32_t v = e >= 0 ? e : -1 - e;
        const std::vector<int32_t> one{v};
        for (int32_t i : e >= 0 ? vals[size_t(v)].in : one)
            if (vals[size_t(i)].leaf >= 0 && !queued[size_t(i)]) {
                queued[size_t(i)] = 1;
                q.push_back(i);
            }
    }
    // slots, loads ahead, waits.  Row loads complete in the order they were
    // issued, stores in any order relative to them: to know a load finished,
    // wait until at most as many operations are outstanding as loads were
    // issued after it (whatever the stores do, the load is then done)
    std::vector<int32_t> slot_of(V, -1), seq_of(V, -1);
    std::vector<int32_t> free_slots;
    for (int32_t sl = kStreamMaxSlots; sl-- > 0;) free_slots.push_back(sl);
    int32_t seq = 0, done = 0, top = 0;  // loads issued, loads finished; slots used
    size_t qi = 0, qused = 0;
    std::vector<uint32_t> loads;  // entries of the load record being built
    auto put = [&](const std::vector<uint32_t>& rec) {
        if (w.size() % 64 + rec.size() > 64) w.resize((w.size() + 63) / 64 * 64, 0u);
        w.insert(w.end(), rec.begin(), rec.end());
    };
    auto flush = [&]() {
        if (loads.empty()) return;
        std::vector<uint32_t> rec{kResLoad | uint32_t(loads.size()) << 8};
        rec.insert(rec.end(), loads.begin(), loads.end());
        put(rec);
        loads.clear();
    };
    auto alloc = [&]() {
        if (free_slots.empty()) return -1;
        const int32_t sl = free_slots.back();
        free_slots.pop_back();
        top = std::max(top, sl + 1);
        return sl;
    };
    auto load_next = [&]() {
        const int32_t v = q[qi];
        const int32_t sl = alloc();
        if (sl < 0) return false;
        slot_of[size_t(v)] = sl;
        seq_of[size_t(v)] = seq++;
        loads.push_back(uint32_t(sl) | uint32_t(vals[size_t(v)].leaf) << 8);
        if (loads.size() == 63) flush();
        ++qi;
        return true;
    };
    auto ready = [&](int32_t v) {  // wait for v's load when still in flight
        if (vals[size_t(v)].leaf < 0 || seq_of[size_t(v)] < done) return;
        flush();
        put({kResWait | uint32_t(std::min(255, seq - seq_of[size_t(v)] - 1)) << 8});
        done = seq_of[size_t(v)] + 1;
    };
    auto release = [&](int32_t v) {
        if (--uses[size_t(v)] == 0) free_slots.push_back(slot_of[size_t(v)]);
    };
    auto store = [&](int32_t v, const std::vector<int32_t>& to) {
        for (size_t i0 = 0; i0 < to.size(); i0 += 126) {
            const size_t c = std::min<size_t>(126, to.size() - i0);
            std::vector<uint32_t> rec((c + 1) / 2 + 1, 0u);
            rec[0] = kResPut | uint32_t(c) << 8 | uint32_t(slot_of[size_t(v)]) << 16;
            for (size_t j = 0; j < c; ++j) rec[1 + j / 2] |= uint32_t(to[i0 + j]) << (16 * (j % 2));
            flush();
            put(rec);
        }
    };
    std::vector<std::pair<int32_t, int32_t>> later;  // stores held back
    for (int32_t e : events) {
        const int32_t v = e >= 0 ? e : -1 - e;
        const std::vector<int32_t> one{v};
        const std::vector<int32_t>& in = e >= 0 ? vals[size_t(v)].in : one;
        for (int32_t i : in)
            if (vals[size_t(i)].leaf >= 0 && seq_of[size_t(i)] < 0) {
                while (seq_of[size_t(i)] < 0)
                    if (!load_next()) return false;
            }
        // one wait, for the input loaded last
        int32_t last = -1;
        for (int32_t i : in) {
            if (vals[size_t(i)].leaf >= 0 && qused < q.size() && q[qused] == i) ++qused;
            if (vals[size_t(i)].leaf >= 0 && (last < 0 || seq_of[size_t(i)] > seq_of[size_t(last)])) last = i;
        }
        if (last >= 0) ready(last);
        if (e >= 0) {  // the fold; its slot: an input's that dies here, else a free one
            const std::vector<int32_t>& x = vals[size_t(v)].in;
            for (int32_t i : x) release(i);
            int32_t sl = -1;
            for (int32_t i : x)
                if (uses[size_t(i)] == 0) {
                    sl = slot_of[size_t(i)];
                    break;
                }
            if (sl >= 0) {
                free_slots.erase(std::find(free_slots.begin(), free_slots.end(), sl));
            } else if ((sl = alloc()) < 0) {
                return false;
            }
            slot_of[size_t(v)] = sl;
            std::vector<uint32_t> rec;
            if (x.size() == 2) {
                rec.push_back(kResAdd2 | uint32_t(slot_of[size_t(x[0])]) << 8 |
                              uint32_t(slot_of[size_t(x[1])]) << 16 | uint32_t(sl) << 24);
            } else {
                rec.assign(1 + (x.size() + 3) / 4, 0u);
                rec[0] = kResFold | uint32_t(x.size()) << 8 | uint32_t(sl) << 16;
                for (size_t j = 0; j < x.size(); ++j)
                    rec[1 + j / 4] |= uint32_t(slot_of[size_t(x[j])]) << (8 * (j % 4));
            }
            flush();
            put(rec);
        } else {  // its stores, but not into a buffer whose row is still to load
            std::vector<int32_t> now;
            for (int32_t b : puts[size_t(v)]) {
                const int32_t l = leaf_of[size_t(b)];
                if (l >= 0 && seen[size_t(l)] && seq_of[size_t(l)] < 0) {
                    later.push_back({v, b});
                    ++uses[size_t(v)];
                } else {
                    if (l >= 0 && seen[size_t(l)]) ready(l);
                    now.push_back(b);
                }
            }
            if (!now.empty()) store(v, now);
            release(v);
        }
        while (qi < q.size() && qi - qused < size_t(kStreamAhead) && free_slots.size() > kStreamReserve)
            if (!load_next()) return false;
    }
    for (const auto& vb : later) {
        ready(leaf_of[size_t(vb.second)]);
        store(vb.first, {vb.second});
        release(vb.first);
    }
    flush();
    nslots = top;
    nload = int64_t(q.size());
    nstore = 0;
    for (size_t v = 0; v < V; ++v)
        if (seen[v]) nstore += int64_t(puts[v].size());
    return true;
}

// The streamed form of sliced run `sd` (stream_kernel): per segment some step
// covers, its streamed program; one unit per 1 KiB tile of such a segment.
// Leaves `sd` in its plain form when a program cannot be built or a table
// would overflow.
static void build_streamed(const Plan& p, const ExecState& ex, SliceDesc& sd) {
    if (p.n > kStreamMaxN || sd.nseg < 1) return;
    const int64_t VEC = 16 / p.esize;
    const size_t nseg = size_t(sd.nseg);
    auto seg_of = [&](int64_t x) {
        return size_t(std::lower_bound(sd.cuts.begin(), sd.cuts.end(), x) - sd.cuts.begin());
    };
    std::vector<std::vector<const XStep*>> steps(nseg);
    for (int32_t q = sd.p0; q < sd.p0 + sd.nphases; ++q)
        for (const XStep& x : ex.phases[size_t(q)].steps) {
            if (x.end <= x.begin) continue;
            for (size_t sg = seg_of(x.begin); sg < seg_of(x.end); ++sg) steps[sg].push_back(&x);
        }
    std::vector<uint32_t> prog;
    std::vector<int32_t> rec_off(nseg, -1), rec_len(nseg, 0);
    int32_t slots = 1;
    int64_t bytes = 0;
    for (size_t sg = 0; sg < nseg; ++sg) {
        if (steps[sg].empty()) continue;
        std::vector<uint32_t> w;
        int32_t sl = 0;
        int64_t nl = 0, ns = 0;
        if (!encode_stream(steps[sg], p.n, w, sl, nl, ns)) return;
        slots = std::max(slots, sl);
        bytes += (nl + ns) * (sd.cuts[sg + 1] - sd.cuts[sg]) * p.esize;
        rec_off[sg] = int32_t(prog.size());
        rec_len[sg] = int32_t(w.size());
        prog.insert(prog.end(), w.begin(), w.end());
        if (prog.size() > size_t(INT32_MAX)) return;
    }
    const int64_t te = int64_t(64) * VEC;
    std::vector<int2> tiles;
    std::vector<ResUnit> units;
    for (size_t sg = 0; sg < nseg; ++sg) {
        if (rec_off[sg] < 0) continue;
        const int64_t len = sd.cuts[sg + 1] - sd.cuts[sg];
        for (int64_t t = 0; t * te < len; ++t) {
            tiles.push_back(make_int2(int(sg), int(t)));
            ResUnit u{};
            u.lo = sd.cuts[sg] + t * te;
            u.nv = int32_t(std::min(te, sd.cuts[sg + 1] - u.lo) / VEC);
            u.off = rec_off[sg];
            u.nw = rec_len[sg];
            u.alias = -1;
            units.push_back(u);
        }
    }
    int32_t max_nw = 0;
    for (const int32_t l : rec_len) max_nw = std::max(max_nw, l);
    // LDS of a workgroup: slots, pointers and program, two workgroups a
    // compute unit at most
    if (units.empty() || int64_t(units.size()) > kMaxBlocks ||
        int64_t(slots) * 1024 + int64_t(p.n) * 8 + int64_t(max_nw) * 4 > kLdsBytesPerCU / 2)
        return;
    sd.resident = true;
    sd.streamed = true;
    sd.slots = slots;
    sd.max_nw = max_nw;
    sd.res_waves = kStreamWaves;
    sd.runits = std::move(units);
    sd.prog = std::move(prog);
    sd.rec_off = std::move(rec_off);
    sd.tiles = std::move(tiles);
    sd.tile_elems = te;
    sd.nunits = int64_t(sd.tiles.size());
    sd.res_bytes = bytes;
}

// The resident form of sliced run `sd` (resident_kernel): per segment some
// step covers, the records of the steps covering it in phase order, the
// buffers whose first touch in the run reads them and the buffers the run
// writes there; one unit per 64 vectors of such a segment.  Leaves `sd` in
// its plain form when the plan has more than kResMaxN buffers or a table
// would overflow.
static void build_resident(const Plan& p, const ExecState& ex, SliceDesc& sd) {
    if (p.n > kResMaxN) {
        build_streamed(p, ex, sd);
        return;
    }
    if (sd.nseg < 1) return;
    const int64_t VEC = 16 / p.esize;
    const size_t nseg = size_t(sd.nseg);
    auto seg_of = [&](int64_t x) {
        return size_t(std::lower_bound(sd.cuts.begin(), sd.cuts.end(), x) - sd.cuts.begin());
    };
    std::vector<std::vector<const XStep*>> steps(nseg);
    // per segment: buffers touched, read before any write, written
    std::vector<uint64_t> seen(nseg, 0), load(nseg, 0), store(nseg, 0);
    for (int32_t q = sd.p0; q < sd.p0 + sd.nphases; ++q) {
        for (const XStep& x : ex.phases[size_t(q)].steps) {
            if (x.end <= x.begin) continue;
            const int k = int(x.srcs.size()), nd = int(x.dsts.size());
            if (k < 1 || nd < 1 || k > kResMaxN || nd > kResMaxN) return;
            uint64_t rd = 0, wr = 0;
            for (int32_t b : x.srcs) rd |= uint64_t(1) << b;
            for (int32_t b : x.dsts) wr |= uint64_t(1) << b;
            for (size_t sg = seg_of(x.begin); sg < seg_of(x.end); ++sg) {
                load[sg] |= rd & ~seen[sg];
                seen[sg] |= rd | wr;
                store[sg] |= wr;
                steps[sg].push_back(&x);
            }
        }
    }
    std::vector<std::vector<uint32_t>> recs(nseg);
    std::vector<std::vector<uint8_t>> alias(nseg);
    for (size_t sg = 0; sg < nseg; ++sg)
        if (!steps[sg].empty()) encode_segment(steps[sg], recs[sg], alias[sg]);
    std::vector<uint32_t> prog;
    std::vector<int32_t> rec_off(nseg, -1), alias_off(nseg, -1);
    for (size_t sg = 0; sg < nseg; ++sg) {
        if (recs[sg].empty()) continue;
        rec_off[sg] = int32_t(prog.size());
        prog.insert(prog.end(), recs[sg].begin(), recs[sg].end());
        if (std::any_of(alias[sg].begin(), alias[sg].end(), [](uint8_t a) { return a != 0xFF; })) {
            alias_off[sg] = int32_t(prog.size());
            for (size_t i = 0; i < 64; i += 4)
                prog.push_back(uint32_t(alias[sg][i]) | uint32_t(alias[sg][i + 1]) << 8 |
                               uint32_t(alias[sg][i + 2]) << 16 | uint32_t(alias[sg][i + 3]) << 24);
        }
        if (prog.size() > size_t(INT32_MAX)) return;
    }
    const int64_t te = int64_t(64) * VEC;
    std::vector<int2> tiles;
    std::vector<ResUnit> units;
    int64_t bytes = 0;
    for (size_t sg = 0; sg < nseg; ++sg) {
        if (recs[sg].empty()) continue;
        const int64_t len = sd.cuts[sg + 1] - sd.cuts[sg];
        bytes += int64_t(__builtin_popcountll(load[sg]) + __builtin_popcountll(store[sg])) * len * p.esize;
        for (int64_t t = 0; t * te < len; ++t) {
            tiles.push_back(make_int2(int(sg), int(t)));
            ResUnit u{};
            u.lo = sd.cuts[sg] + t * te;
            u.load = load[sg];
            u.store = store[sg];
            u.nv = int32_t(std::min(te, sd.cuts[sg + 1] - u.lo) / VEC);
            u.off = rec_off[sg];
            u.nw = int32_t(recs[sg].size());
            u.alias = alias_off[sg];
            units.push_back(u);
        }
    }
    if (units.empty() || int64_t(units.size()) > kMaxBlocks) return;
    sd.resident = true;
    sd.res_waves = res_waves(p.n, int64_t(units.size()));
    sd.runits = std::move(units);
    sd.prog = std::move(prog);
    sd.rec_off = std::move(rec_off);
    sd.tiles = std::move(tiles);
    sd.tile_elems = te;
    sd.nunits = int64_t(sd.tiles.size());
    sd.res_bytes = bytes;
}

// Per executed phase, what the choice of sliced runs needs: whether every
// step boundary is 16-byte aligned, the bytes written and moved, the most
// steps covering one element position, and the predicted phase-launch time.
struct PhaseCost {
    bool aligned = true;
    int64_t written = 0, read = 0, bytes = 0, cover = 0;
    int32_t kmax = 0, dmax = 0;
    uint64_t touched = 0;  // buffers the phase touches (n <= kResMaxN)
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
    for (const LaunchDesc& L : ex.launches)
        pc[size_t(L.xphase)].t_launch += kLaunchNs + std::max(kKernelMinNs, double(L.hbm) / kBytesPerNs);
    return pc;
}

// Sliced runs for AR_OPT_SLICE = 2: phases [a, b), each aligned, writing at
// most kKeepBytes and moving at most kSliceMaxBytes, chosen to minimise the
// predicted time, each in its plain or (AR_OPT_RESIDENT, n <= kResMaxN) its
// resident form, whichever is predicted faster.  A run of one phase only
// pays off when it replaces several launches.
struct Run {
    int32_t a, b;
    bool resident;
};

static std::vector<Run> choose_runs(const Plan& p, const ExecState& ex,
                                    const std::vector<PhaseCost>& pc) {
    const double per_src = p.dtype == AR_BF16 ? kStepNsPerSrcBF16 : kStepNsPerSrcF32;
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
            plain_ok = plain_ok && c.written <= kKeepBytes && c.bytes <= kSliceMaxBytes;
            if (!plain_ok && !res_ok) break;
            body += std::max({double(c.cover) * (kStepNs + per_src * c.kmax + kStepNsPerDst * c.dmax),
                              stretch * double(c.read) / kBytesPerNs,
                              double(c.written) / kBytesPerNs});
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
            if (b - a == 1 && nl[size_t(a)] < 2) continue;
            double t = plain_ok ? kLaunchNs + body : std::numeric_limits<double>::infinity();
            bool res = false;
            if (res_ok) {
                const double rows = 2.0 * double(__builtin_popcountll(touched));
                const double t_waves = rounds * (kResRowNs / W * rows + chain);
                const double t_bytes = rows * double(p.N) * p.esize / kBytesPerNs;
                const double t_res = kLaunchNs + std::max(t_waves, t_bytes) +
                                     kResOverlap * std::min(t_waves, t_bytes);
                if (t_res < t) {
                    t = t_res;
                    res = true;
                }
            }
            if (best[size_t(a)] + t < best[size_t(b)]) {
                best[size_t(b)] = best[size_t(a)] + t;
                from[size_t(b)] = a;
                res_of[size_t(b)] = res;
            }
        }
    }
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

ExecState* exec_state(Plan& p) {
    if (!p.exec) {
        ExecState* ex = new ExecState();
        try {
            ex->phases = exec_phases(p, p.fuse != 0);
            build_launches(p, *ex);
            std::vector<Run> runs;
            if (p.slice == 1 && !ex->phases.empty()) {
                runs.push_back({0, int32_t(ex->phases.size()), p.resident != 0});
            } else if (p.slice == 2) {
                runs = choose_runs(p, *ex, phase_costs(p, *ex));
            }
            std::vector<int32_t> slice_of(ex->phases.size(), -1);
            for (const Run& r : runs) {
                SliceDesc sd = build_slice(p, *ex, r.a, r.b);
                if (!sd.ok) continue;  // phase launches for these phases
                if (r.resident) build_resident(p, *ex, sd);
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
