// Resident and streamed programs of sliced runs (resident_kernel and
// stream_kernel, encodings in resident.hpp): per segment of a run, the
// records of its steps, the rows to load and to store or the slots, loads,
// waits and stores, and one unit per tile.  Host only.
#include <algorithm>
#include <functional>
#include <vector>

#include "exec_state.hpp"

namespace arp {

// Wavefronts per resident workgroup: four issue a tile's row loads and
// stores in parallel, which pays when LDS already limits a compute unit to
// at most eight tiles (32 waves) or when there are too few tiles to fill the
// chip; otherwise one wave per tile lets a unit hold more tiles.
int32_t res_waves(int32_t n, int64_t units) {
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
// waves of a streamed workgroup (the kernel is written for 1 or 4; one wave
// owning the whole tile measured the same as four owning a quarter each, and
// the executor launches four)
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
void build_resident(const Plan& p, const ExecState& ex, SliceDesc& sd) {
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

}  // namespace arp
