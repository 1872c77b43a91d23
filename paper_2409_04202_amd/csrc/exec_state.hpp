// Host-side state of the executor, shared by its translation units: the
// executed phases after the rewrites (rewrite.cpp), their launches and
// sliced runs (schedule.cpp), the resident and streamed programs
// (programs.cpp), and the per-device state and launching (exec.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "resident.hpp"
#include "../../include/ar_plan.h"
#include "plan.hpp"

namespace arp {


constexpr int kCache = 4;               // buffer sets whose step records are kept per device
// Wave tiles are halved (down to one iteration of the kernel's loop) until a
// launch has kMinUnits of them, kMinUnitsReduce for a launch that folds two
// or more sources: short reduce launches ramp up and drain in a sizeable
// part of their time, and finer tiles shorten the drain (measured: the bf16
// tree (8, 8, 8)'s 288 MiB level-0 fold 5.05 -> 5.83 TB/s, the tree (8, 8)'s
// 144 MiB level-1 fold 5.11 -> 5.46 TB/s; launches already past 16384 tiles
// are unchanged).
constexpr int64_t kMinUnits = 2048;
constexpr int64_t kMinUnitsReduce = 16384;
// A launch of at least kFineTileMinBytes with fewer than kMinUnits tiles at
// the smallest full-pass tile (64 lanes x U vectors per source) halves its
// tile further, down to one vector per lane, until it has kMinUnits (not
// for copies reading a range several times: their XCD tables lost with
// smaller tiles, the tree (8, 4) at 1 MiB per processor +50 %).  Measured
// as written: Ring n = 64 at 1M elements 0.77 -> 0.55 ms (f32) and
// 0.60 -> 0.44 ms (bf16), Ring n = 8 and RHD n = 8 at 1 MiB per processor
// -29 % and -27 %.
constexpr int64_t kFineTileMinBytes = int64_t(2) << 20;
// A 2-source launch of at least kWideBytes with nontemporal loads and stores
// and a full kcfg tile (64 lanes x kWideU vectors) runs the wide instance of
// the phase kernel (kWideU vectors per lane and source in one pass); so does
// an 8-source launch of 4-byte elements of that size with nontemporal loads
// (kWideU8 vectors per lane and source: 198 -> 196 us for the (8, 8) tree's
// 1.1 GiB first level; bf16 folds ran 3 % slower with it).
constexpr int64_t kWideBytes = int64_t(512) << 20;
// A runtime-source-count launch (a fan-in without an unrolled kernel)
// moving less than kRtGroupMaxBytes keeps the loads of kRtGroup sources in
// flight together; larger ones load one source at a time (measured: k = 24
// at 1 MiB per processor 22.3 -> 16.4 us, k = 32 at 64 MiB 0.372 ms one
// at a time against 0.400 grouped).
constexpr int64_t kRtGroupMaxBytes = int64_t(512) << 20;
constexpr int64_t kMaxBlocks = int64_t(1) << 24;
// Cache policy per launch (measured on MI355X).  Launches moving less than
// kNtBytes keep everything cached.  Larger ones load nontemporally unless a
// source range is read by more than one step of the launch (then the repeated
// reads hit the cache), and store nontemporally unless the next phase reads
// what they write and it is at most kKeepBytes, small enough to stay in the
// 256 MiB last-level cache until then.
constexpr int64_t kNtBytes = int64_t(64) << 20;
constexpr int64_t kKeepBytes = int64_t(256) << 20;
// A fold launch keeps its stores cached up to kKeepBytesFold: RHD's second
// halving launch (512 MiB written, read by the third) ran 271 -> 254 us with
// cached stores, and the third 126 -> 124 us, part of its reads hitting the
// cache; copy launches of that size ran slower with cached stores (the
// 1 GiB doubling copy 164 -> 167 us).
constexpr int64_t kKeepBytesFold = int64_t(512) << 20;
// A fold launch whose previous phase kept all its stores cached and wrote
// at most kWarmBytes loads through the cache even when large: the two-level
// tree's level-1 fold (8 sources, 4 MiB f32 each, reading the 128 MiB that
// level 0 wrote) took the whole as-written plan 0.403 -> 0.395 ms; copies
// under the same rule ran slower (RHD's first doubling copy).
constexpr int64_t kWarmBytes = int64_t(256) << 20;
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
// consecutive executed phases may become one plain sliced launch when every
// phase in it writes at most kKeepBytes (what one phase hands to the next
// would stay in the last-level cache with phase launches as well) and moves
// at most kSliceMaxBytes; a resident run (below) keeps what its phases hand
// on in LDS and takes phases of any size.  The runs are chosen by dynamic programming over the phases
// with a cost model fitted to MI355X measurements (back-to-back launches, no
// events between them):
//  * bytes move at kBytesPerNs, or at kCachedBytesPerNs when the plan's whole
//    footprint n * N * e fits the kCacheBytes last-level cache;
//  * a phase launch costs kPhaseLaunchNs plus its HBM traffic, at least
//    kKernelMinNs per dependent round of loads (one dependent load and store
//    through memory; a runtime-source-count fold loads its k sources in
//    ceil(k / rt_group) rounds);
//  * a sliced launch costs kLaunchNs plus, per phase, the largest of its
//    dependent chain, its read time and its write time.  The chain is the
//    most steps covering one element position, which a wavefront runs one
//    after the other, at kStepNs + k * kStepNsPerSrc{F32,BF16} +
//    d * kStepNsPerDst each (k, d = the phase's largest source and
//    destination counts); the reads are stretched by kMinSliceWaves / waves
//    when the slice has fewer wave tiles than that (too few loads in flight
//    to reach full bandwidth).
// The constants of these forms and of the resident form (below) were fitted
// together, in log error, to 151 plans (Ring, RHD, co-located PS, 2- and
// 3-level trees, n = 8 to 512, 4K to 1M elements, fp32 and bf16) each timed
// as phase launches, as one plain sliced launch and (n <= 64) as one
// resident launch: the prediction error of the phase launches 59 -> 11 %
// mean, the form the model ranks first within 5 % of the fastest in 141 of
// the 151 plans (from 114).  kBytesPerNs comes from the HBM-bound
// workloads, whose footprints exceed the cache.  Terms the fit put at zero
// (per-destination step costs, the resident per-row cost, sharing between
// workgroups) are kept, at 0.
constexpr double kLaunchNs = 2200.0;
constexpr double kPhaseLaunchNs = 1550.0;
constexpr double kKernelMinNs = 1750.0;
constexpr double kBytesPerNs = 5500.0;
constexpr double kCachedBytesPerNs = 6450.0;
constexpr int64_t kCacheBytes = int64_t(256) << 20;
constexpr double kStepNs = 265.0;
constexpr double kStepNsPerSrcF32 = 205.0;
constexpr double kStepNsPerSrcBF16 = 300.0;
constexpr double kStepNsPerDst = 0.0;
constexpr double kMinSliceWaves = 400.0;
constexpr int64_t kSliceMaxBytes = int64_t(512) << 20;
// A sliced run of one phase replacing that phase's only launch is taken only
// when predicted to cost at most this fraction of the launch: for one phase
// the estimate above is optimistic (co-located PS n = 16 at 2^18 fp32 and at
// 2^20 bf16 run slower sliced than predicted); 0.75 picked best over the
// co-located PS plans of the fit (n = 16 to 64, sliced where a 32- or
// 64-source fold into as many buffers runs as one launch at 2^18).
constexpr double kSingleRunGain = 0.75;
// A sliced run may instead run resident (resident_kernel, AR_OPT_RESIDENT):
// a workgroup of W waves (res_waves in programs.cpp) per 64 vectors of a
// segment, the plan's n <= kResMaxN buffers in LDS rows of 1 KiB.  Its
// predicted time is kLaunchNs plus the larger of its HBM traffic (each row
// read and written once) and its workgroups' time, plus
// kResOverlap times the smaller (with few workgroups per compute unit the
// two overlap only in part).  A workgroup takes kResRowNs / W per row
// loaded or stored, and per step of its chain kResChainNs for a 2-source,
// 1-destination step that is the only one on its positions in its phase and
// follows another such phase of the run (these form chain records),
// kResFastNs for other one-word records (two sources or a copy, one
// destination), or kResStepNs + k * kResStepNsPerSrc + d * kResStepNsPerDst
// (d = 1 in the run's last phase, whose further destinations the store pass
// writes through the alias table).  Workgroups run kResWavesPerCU (one
// wave) or 8 (four waves) per compute unit at a time, or fewer when their
// LDS rows do not fit (kLdsBytesPerCU), and those sharing a unit (when there
// are more tiles than units) slow each other by kResShare per extra one.
constexpr double kResRowNs = 0.0;
constexpr double kResFastNs = 275.0;
constexpr double kResChainNs = 77.0;
constexpr double kResStepNs = 240.0;
constexpr double kResStepNsPerSrc = 50.0;
constexpr double kResStepNsPerDst = 0.0;
constexpr double kResShare = 0.0;
constexpr double kResOverlap = 0.45;
// A resident run that does not start at the first executed phase costs
// kResAfterLaunchNs more: measured, its time hardly shrinks with the phases
// left to the launches before it (RHD n = 32 at 2^16 fp32: the first phase
// as a launch, then the rest resident, 15.2 us; all of it resident 11.1 us;
// RHD n = 48 at 2^13, two phases as launches, 16.1 against 14.0 us), while
// the model's chain terms would have it shrink; with fan-in 4 trees over 64
// buffers at 4K-16K elements the split still pays (9.9 against 11.4 us).
constexpr double kResAfterLaunchNs = 3000.0;
constexpr int64_t kResWavesPerCU = 16;
constexpr int64_t kLdsBytesPerCU = int64_t(160) << 10;
constexpr int64_t kNumCUs = 256;
constexpr int64_t kNumXCDs = 8;         // compute dies, each with its own L2
// A plan of more than kResMaxN buffers may run as one streamed launch
// (stream_kernel) under AR_OPT_SLICE = 2 as well, when that is predicted
// below kStreamGain of the runs chosen above.  Its workgroups each run one
// unit's program, one record after the other, as many at a time as LDS
// holds (slots, buffer pointers and the longest unit program per
// workgroup): kLaunchNs + rounds * words * kStreamWordNs, rounds = units
// over the workgroups that fit.  Measured on MI355X (48 plans, n = 96-512,
// 4K-1M elements): 120-155 ns per word for Ring and RHD, 77-110 for trees;
// the streamed form beat the other choice only on Ring (n = 128 and 256 up
// to 256K fp32 elements, n = 128 up to 1M bf16: 0.45-0.91 of its time).
// The prediction of those runs was low (88-215 us against 101-408
// measured), so the streamed form is taken whenever predicted faster
// (kStreamGain 1): on the 48 plans it was then picked 7 times, each a win.
constexpr double kStreamWordNs = 145.0;
constexpr double kStreamGain = 1.0;
// With more than kResMaxN buffers (beyond the plans the model was fitted
// on) a plain sliced run leaves out phases whose steps store to at least
// kSplitMinDst buffers over ranges shorter than kSlicedManyDstMinBytes: a
// wave of the sliced kernel stores each such step alone, mostly with idle
// lanes, where their own launch runs split.  Measured: RHD n = 96-256 at
// 4K-32K fp32 elements took 1.2-1.7 times as long with such a run as with
// phase launches.
constexpr int64_t kSlicedManyDstMinBytes = 4096;
// Copy launches whose steps read a range several times deal their tiles to
// XCDs by source range (xcd_tiles in schedule.cpp) when a step has at most
// this many tiles.
constexpr int64_t kXcdMaxTiles = 64;

// A launch of fewer than kMinUnits wave tiles whose steps store to at least
// kSplitMinDst destinations is split (a workgroup of kSplitWaves per tile,
// see split_tile) when it moves less than kNtBytes or stores to at least
// kSplitWideDst destinations per source.  Measured on MI355X against the
// same launches unsplit (both placed by position): under 64 MiB every
// split launch was faster (the bf16 tree (8, 8, 8)'s level-2 reduce 13.8 ->
// 12.2 us, Ring n = 64's last halving step at 2^16 fp32 22.1 -> 9.3 us,
// 16-source folds 12.0 -> 10.5 us); above, Ring n = 64 at 2^20 (32
// destinations per source) 59.6 -> 49.6 us, but the 8-source folds into 64
// buffers of the bf16 trees at 2^20 ran 28-30 us unsplit against 32-34.
constexpr int32_t kSplitMinDst = 16;
constexpr int32_t kSplitWideDst = 16;
// Launches moving at most kAffinityMaxBytes, and split launches, place their
// tiles on XCDs by element position (affinity_tiles in schedule.cpp, xcd_of
// below), so that what one such launch writes is read by the next on the
// XCD whose L2 holds it.  Measured on MI355X: the bf16 tree (8, 8, 8)'s split level-2
// reduce (sources written by the 36 MiB level-1 reduce) 19.8 -> 12.5 us;
// phase launches of the tree (8, 8) at 2^16 fp32 and Ring n = 4 at 2^16,
// 14-32 % less per AllReduce; but with a limit of 512 MiB the tree (8, 8)'s
// 144 MiB level-1 reduce ran 27 -> 31 us.  Launches of one or two sources
// moving at least kAffinityBigBytes and reading every range once are placed
// so too: RHD as written (n = 8, 2^26 fp32) 1.531 -> 1.503 ms, each of its
// halving folds and doubling copies 1-4 % faster; the 16-source fold placed
// so left its own time unchanged and slowed the AllGather copies after it
// (182 -> 189 us), which read its output from other XCDs.
constexpr int64_t kAffinityMaxBytes = int64_t(64) << 20;
constexpr int64_t kAffinityBigBytes = int64_t(512) << 20;

// XCD of a tile starting at element e of N: each XCD owns a contiguous
// 1/kNumXCDs of every buffer's element range.  Launches with an affinity
// table place their tiles this way, so a launch reading (or overwriting)
// what the launch before it wrote finds it in its own XCD's L2 rather than
// in another's (the XCDs' L2s are kept coherent with each other, and a line
// another XCD holds is slow to read or overwrite), and each XCD gets an
// equal share of a phase that covers the whole vector.  Shared with the
// host-side check.
inline int64_t xcd_of(int64_t e, int64_t N) {
    return N > 0 ? std::min<int64_t>(e * kNumXCDs / N, kNumXCDs - 1) : 0;
}

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
    int32_t rt_group;        // runtime-k kernel: sources with loads in flight together
    int32_t dsplit;          // waves per tile (split_tile), 1: one
    int32_t affinity;        // 1: the tile table places tiles by xcd_of
    int32_t wide;            // 1: the wide 2-source instance (kWideU per pass)
    int64_t bytes;           // (k + destinations) * len * e over the steps
    int64_t hbm;             // predicted HBM traffic: bytes, less the repeated
                             // reads of a range by the launch's copies
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
    ResUnit* runits = nullptr;   // resident units and records, all slices concatenated
    uint32_t* prog = nullptr;
    PtrEntry cache[kCache];
    uint64_t clock = 0;
};

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
    // resident form (resident_kernel): one ResUnit per wave and, per
    // segment, its step records in `prog` (rec_off[s]: first word, -1 for a
    // segment no step covers); `tiles` and `tile_elems` are then the
    // resident kernel's tiles (one vector per lane), unit i = tiles[i]
    bool resident = false;
    int32_t res_waves = 1;       // wavefronts per resident workgroup (1 or 4)
    // streamed form (stream_kernel, plans with more than kResMaxN buffers):
    // resident with `slots` LDS slots of 1 KiB per workgroup and load, wait
    // and store records in `prog`; the units' row masks are then zero
    bool streamed = false;
    int32_t slots = 0;
    int32_t max_nw = 0;          // words of the longest unit program (in LDS)
    std::vector<ResUnit> runits;
    std::vector<uint32_t> prog;
    std::vector<int32_t> rec_off;
    int64_t runit_base = 0, prog_base = 0;
    int64_t res_bytes = 0;       // bytes the resident launch loads and stores
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
    int64_t rec_words = 0;       // words of all records; the n buffer
                                 // pointers follow them (resident launches)
    std::vector<SliceDesc> slices;
    std::vector<Stage> stages;   // the launches for 16-byte aligned buffers
    std::vector<DevState*> dev;  // indexed by device ordinal
    uint64_t serial = 0;         // unique per executor state ever built
    // ar_plan_execute_noalloc: the tables and step records laid out as in
    // the scratch array (built on its first call with this state)
    std::vector<uint64_t> img;
    int64_t img_off[8] = {};     // byte offsets: tiles, cuts, sched_off,
                                 // sched, stiles, runits, prog, records
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

// Template source count of the phase kernel for k sources (0: read at run
// time).
int kernel_k(int32_t k);

// Executed phases of a plan, after the rewrites when `fuse` (rewrite.cpp).
std::vector<XPhase> exec_phases(const Plan& p, bool fuse);

// Is every executed phase free of hazards?  (rewrite.cpp)
bool exec_phases_hazard_free(const std::vector<XPhase>& ph, int32_t n, std::string& why);

// The plan's executor state under its current options, built on first use
// (schedule.cpp).  Host only.
ExecState* exec_state(Plan& p);
// Wavefronts per resident workgroup for a plan of n buffers and `units` tiles
// (programs.cpp).
int32_t res_waves(int32_t n, int64_t units);
// The resident (n <= kResMaxN) or streamed form of sliced run `sd`, in place;
// `sd` stays plain when its program cannot be built (programs.cpp).
void build_resident(const Plan& p, const ExecState& ex, SliceDesc& sd);

}  // namespace arp
