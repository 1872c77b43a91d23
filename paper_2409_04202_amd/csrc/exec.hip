// Executor: turns a plan's executed phases into kernel launches on a HIP
// stream, plus the timing API and the executor options.
//
// An execution is a list of stages (schedule.cpp): phase launches, where the
// steps of one phase with the same source count k (copies are k = 1) run as
// one launch of phase_kernel<dtype, k, aligned, cache mode>, and sliced
// launches of runs of phases (sliced_kernel, or resident_kernel).  Kernels
// read each step as a record holding its range and its resolved buffer
// pointers (StepHead); the records of a buffer set, followed by its n buffer
// pointers, are built on the host and uploaded once, and a small per-plan
// cache keeps them per device, so repeated executes on the same buffers
// launch kernels only.  The tile, sliced and resident tables are uploaded on
// the first execute on a device.  Buffers that are not 16-byte aligned run
// every phase as its phase launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <tuple>
#include <new>
#include <string>
#include <vector>

#include "exec_state.hpp"
#include "internal.hpp"

namespace arp {

namespace {

std::string hip_msg(const char* what, hipError_t e) {
    return std::string(what) + ": " + hipGetErrorName(e) + " (" +
           hipGetErrorString(e) + ")";
}

}  // namespace

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
    if (d->runits) (void)hipFree(d->runits);
    if (d->prog) (void)hipFree(d->prog);
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

// The sliced launches' tables of all slices, concatenated (each slice
// indexes them from its *_base offsets).
struct SliceTables {
    std::vector<int64_t> cuts;
    std::vector<int32_t> soff, sched;
    std::vector<int2> tiles;
    std::vector<ResUnit> runits;
    std::vector<uint32_t> prog;
};

static SliceTables slice_tables(const ExecState& ex) {
    SliceTables t;
    for (const SliceDesc& sd : ex.slices) {
        t.cuts.insert(t.cuts.end(), sd.cuts.begin(), sd.cuts.end());
        t.soff.insert(t.soff.end(), sd.sched_off.begin(), sd.sched_off.end());
        t.sched.insert(t.sched.end(), sd.sched.begin(), sd.sched.end());
        t.tiles.insert(t.tiles.end(), sd.tiles.begin(), sd.tiles.end());
        t.runits.insert(t.runits.end(), sd.runits.begin(), sd.runits.end());
        t.prog.insert(t.prog.end(), sd.prog.begin(), sd.prog.end());
    }
    return t;
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
            const SliceTables t = slice_tables(ex);
            s = upload(&d->cuts, t.cuts, "segment table");
            if (s == AR_OK) s = upload(&d->sched_off, t.soff, "schedule offsets");
            if (s == AR_OK) s = upload(&d->sched, t.sched, "schedule");
            if (s == AR_OK) s = upload(&d->stiles, t.tiles, "slice tiles");
            if (s == AR_OK) s = upload(&d->runits, t.runits, "resident units");
            if (s == AR_OK) s = upload(&d->prog, t.prog, "resident programs");
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

static bool buffers_aligned(void* const* bufs, int32_t n) {
    for (int32_t i = 0; i < n; ++i)
        if (reinterpret_cast<uint64_t>(bufs[i]) & 15) return false;
    return true;
}

// The step records of buffer set bufs[0..n) (see StepHead) followed by the n
// buffer pointers, written to w[0 .. rec_words + n).
static void fill_records(const ExecState& ex, void* const* bufs, int32_t n, uint64_t* w) {
    std::memset(w, 0, size_t(ex.rec_words + n) * sizeof(uint64_t));
    for (size_t i = 0; i < ex.hsteps.size(); ++i) {
        const DevStep& st = ex.hsteps[i];
        uint64_t* r = w + ex.rec_of[i];
        StepHead h{st.begin, st.end, st.k, st.ndst, st.nfree, 0};
        std::memcpy(r, &h, sizeof(h));
        for (int32_t j = 0; j < st.k; ++j)
            r[kRecHead + j] = reinterpret_cast<uint64_t>(bufs[size_t(ex.hidx[size_t(st.src_off + j)])]);
        for (int32_t j = 0; j < st.ndst; ++j)
            r[kRecHead + st.k + j] =
                reinterpret_cast<uint64_t>(bufs[size_t(ex.hidx[size_t(st.dst_off + j)])]);
    }
    for (int32_t i = 0; i < n; ++i) w[ex.rec_words + i] = reinterpret_cast<uint64_t>(bufs[i]);
}

// The step records for buffer set `bufs` on this device (see StepHead),
// followed by the n buffer pointers: from the per-plan cache, or built on
// the host and uploaded on `stream`.
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
    const size_t nb = size_t(ex.rec_words + p.n) * sizeof(uint64_t);
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
    fill_records(ex, bufs.data(), p.n, v->pinned);
    e = hipMemcpyAsync(v->dev, v->pinned, nb, hipMemcpyHostToDevice, stream);
    if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("step record upload", e));
    e = hipEventRecord(v->done, stream);
    if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("hipEventRecord", e));
    v->key = bufs;
    v->valid = true;
    v->stamp = d.clock;
    v->aligned = buffers_aligned(bufs.data(), p.n);
    *out = v;
    return AR_OK;
}

template <int DT, int K>
static void launch_dk(bool vecok, int cm, int64_t blocks, hipStream_t st,
                      const uint64_t* recs, int64_t stride, const int2* tiles,
                      int64_t nunits, int64_t tps, int64_t te, int rtg,
                      int dsplit, int wide) {
    const dim3 block(64 * kcfg(K).WPB);
    if constexpr (K == 2) {
        if (wide && vecok && cm == 3 && dsplit == 1) {  // see kWideBytes
            hipLaunchKernelGGL((phase_kernel<DT, 2, true, 3, kWideU>),
                               dim3(static_cast<uint32_t>(blocks)), block, 0, st, recs, stride,
                               tiles, nunits, tps, te, rtg);
            return;
        }
    }
    if constexpr (K == 8 && DT != DT_BF16) {
        if (wide && vecok && (cm & 1) && dsplit == 1) {  // see kWideBytes
            if (cm & 2)
                hipLaunchKernelGGL((phase_kernel<DT, 8, true, 3, kWideU8>),
                                   dim3(static_cast<uint32_t>(blocks)), block, 0, st, recs,
                                   stride, tiles, nunits, tps, te, rtg);
            else
                hipLaunchKernelGGL((phase_kernel<DT, 8, true, 1, kWideU8>),
                                   dim3(static_cast<uint32_t>(blocks)), block, 0, st, recs,
                                   stride, tiles, nunits, tps, te, rtg);
            return;
        }
    }
    if (dsplit > 1 && vecok) {  // a workgroup per table entry
        // the waves of a workgroup all read the tile's sources: cached loads
        // (with nontemporal ones each wave fetched them from memory again)
        const int64_t ntiles = nunits / dsplit;
        const dim3 grid(static_cast<uint32_t>(ntiles)), sblock(64 * kSplitWaves);
        if (cm & 2)
            hipLaunchKernelGGL((split_kernel<DT, K, 2>), grid, sblock, 0, st, recs, stride, tiles,
                               ntiles, te, rtg);
        else
            hipLaunchKernelGGL((split_kernel<DT, K, 0>), grid, sblock, 0, st, recs, stride, tiles,
                               ntiles, te, rtg);
        return;
    }
    if (dsplit > 1) {  // unaligned buffers: one wave per table entry
        nunits /= dsplit;
        blocks = (nunits + kcfg(K).WPB - 1) / kcfg(K).WPB;
    }
    const dim3 grid(static_cast<uint32_t>(blocks));
#define AR_LAUNCH(V, C)                                                                \
    hipLaunchKernelGGL((phase_kernel<DT, K, V, C>), grid, block, 0, st, recs, stride, \
                       tiles, nunits, tps, te, rtg)
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
                     int64_t nunits, int64_t tps, int64_t te, int rtg,
                     int dsplit, int wide) {
    switch (K) {
        case 1: launch_dk<DT, 1>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te, rtg, dsplit, wide); break;
        case 2: launch_dk<DT, 2>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te, rtg, dsplit, wide); break;
        case 3: launch_dk<DT, 3>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te, rtg, dsplit, wide); break;
        case 4: launch_dk<DT, 4>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te, rtg, dsplit, wide); break;
        case 8: launch_dk<DT, 8>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te, rtg, dsplit, wide); break;
        case 16: launch_dk<DT, 16>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te, rtg, dsplit, wide); break;
        default: launch_dk<DT, 0>(vecok, cm, blocks, st, recs, stride, tiles, nunits, tps, te, rtg, dsplit, wide); break;
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

// Where one execution's device-side tables and step records are: the
// plan's own device state, or the no-allocation entry point's scratch.
struct DevView {
    const int2* tiles;
    const int64_t* cuts;
    const int32_t* sched_off;
    const int32_t* sched;
    const int2* stiles;
    const ResUnit* runits;
    const uint32_t* prog;
    const uint64_t* recs;  // step records, then the n buffer pointers
    bool aligned;          // every buffer 16-byte aligned
};

// Enqueue the launches of one execution on `stream`.
static ar_status launch_all(ar_plan* plan, const ExecState* ex, const DevView& v,
                            hipStream_t stream, ar_timer* timer) {
    const DevView* d = &v;
    ar_status s = AR_OK;
    {
        // sliced launches need 16-byte aligned buffers; otherwise every
        // phase runs as its phase launches
        const bool staged = v.aligned;
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
            if (stg.slice >= 0 && ex->slices[size_t(stg.slice)].streamed) {
                const SliceDesc& sd = ex->slices[size_t(stg.slice)];
                if (sd.res_waves != 4) return fail(AR_ERR_INTERNAL, "streamed launch shape");
                const dim3 grid(static_cast<uint32_t>(sd.nunits)), block(256);
                // the slots, the n buffer pointers, the longest unit program
                const size_t lds = size_t(sd.slots) * 1024 + size_t(plan->n) * 8 + size_t(sd.max_nw) * 4;
                const bool nt = sd.res_bytes > 2 * kKeepBytes;
#define AR_STREAM_K(DT, W, NT)                                                                \
    hipLaunchKernelGGL((stream_kernel<DT, W, NT>), grid, block, lds, stream,                    \
                       v.recs + ex->rec_words, plan->n, sd.slots,                              \
                       d->runits + sd.runit_base, d->prog + sd.prog_base, sd.nunits)
#define AR_STREAM(DT)                                                                         \
    if (nt) AR_STREAM_K(DT, 4, true);                                                         \
    else AR_STREAM_K(DT, 4, false)
                switch (plan->dtype) {
                    case AR_F32: AR_STREAM(DT_F32); break;
                    case AR_I32: AR_STREAM(DT_I32); break;
                    default: AR_STREAM(DT_BF16); break;
                }
#undef AR_STREAM
#undef AR_STREAM_K
            } else if (stg.slice >= 0 && ex->slices[size_t(stg.slice)].resident) {
                const SliceDesc& sd = ex->slices[size_t(stg.slice)];
                const dim3 grid(static_cast<uint32_t>(sd.nunits)), block(64 * sd.res_waves);
                const size_t lds = size_t(plan->n) * 1024;
#define AR_RESIDENT(DT, W, NT)                                                                \
    hipLaunchKernelGGL((resident_kernel<DT, W, NT>), grid, block, lds, stream,                \
                       v.recs + ex->rec_words, plan->n, d->runits + sd.runit_base,           \
                       d->prog + sd.prog_base, sd.nunits)
                // runs moving more than the last-level cache holds stream
                // their rows past it
                const bool nt = sd.res_bytes > 2 * kKeepBytes;
#define AR_RESIDENT_W(DT)                                                                     \
    if (sd.res_waves == 4) {                                                                  \
        if (nt) AR_RESIDENT(DT, 4, true); else AR_RESIDENT(DT, 4, false);                     \
    } else {                                                                                  \
        if (nt) AR_RESIDENT(DT, 1, true); else AR_RESIDENT(DT, 1, false);                     \
    }
                switch (plan->dtype) {
                    case AR_F32: AR_RESIDENT_W(DT_F32); break;
                    case AR_I32: AR_RESIDENT_W(DT_I32); break;
                    default: AR_RESIDENT_W(DT_BF16); break;
                }
#undef AR_RESIDENT_W
#undef AR_RESIDENT
            } else if (stg.slice >= 0) {
                const SliceDesc& sd = ex->slices[size_t(stg.slice)];
                const dim3 grid(static_cast<uint32_t>((sd.nunits + kSliceWPB - 1) / kSliceWPB));
                const dim3 block(64 * kSliceWPB);
#define AR_SLICED(DT)                                                                   \
    hipLaunchKernelGGL((sliced_kernel<DT>), grid, block, 0, stream, v.recs,             \
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
                const uint64_t* recs = v.recs + L.rec_off;
                const int2* tiles = L.tile_off >= 0 ? d->tiles + L.tile_off : nullptr;
                switch (plan->dtype) {
                    case AR_F32:
                        launch_d<DT_F32>(L.kern_k, v.aligned, L.cm, blocks, stream, recs,
                                         L.rec_stride, tiles, L.nunits, L.tiles_per_step,
                                         L.tile_elems, L.rt_group, L.dsplit, L.wide);
                        break;
                    case AR_I32:
                        launch_d<DT_I32>(L.kern_k, v.aligned, L.cm, blocks, stream, recs,
                                         L.rec_stride, tiles, L.nunits, L.tiles_per_step,
                                         L.tile_elems, L.rt_group, L.dsplit, L.wide);
                        break;
                    default:
                        launch_d<DT_BF16>(L.kern_k, v.aligned, L.cm, blocks, stream, recs,
                                          L.rec_stride, tiles, L.nunits, L.tiles_per_step,
                                          L.tile_elems, L.rt_group, L.dsplit, L.wide);
                        break;
                }
            }
            hipError_t he = hipGetLastError();
            if (he != hipSuccess) return fail(AR_ERR_HIP, hip_msg("kernel launch", he));
            s = mark(1);
            if (s != AR_OK) return s;
            if (timer) timer->launch[size_t(timer->count++)] = int32_t(li);
        }
    }
    return AR_OK;
}

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
        const DevView v{d->tiles, d->cuts, d->sched_off, d->sched, d->stiles,
                        d->runits, d->prog, pe->dev, pe->aligned};
        return launch_all(plan, ex, v, stream, timer);
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}

// ------------------------------------------- execution without allocation
//
// ar_plan_execute_noalloc keeps an execution's device-side tables and step
// records in `scratch`, a fixed array of this library on every device (no
// device allocation at any call).  Host code never uses the array's name
// as an address: on a device's first call the device address comes from
// hipGetSymbolAddress with that device current, and is kept per device.
// Calls on one device share the array; the host remembers which executor
// state and buffer set the last call on each device wrote into it and
// copies the tables and records again only when they differ.

static __device__ __align__(256) uint8_t scratch[AR_NOALLOC_MAX_BYTES];

namespace {

struct ScratchDev {
    uint8_t* ptr = nullptr;       // device address of `scratch` on this device
    uint64_t serial = 0;          // executor state whose tables it holds
    std::vector<void*> bufs;      // buffer set whose records it holds
};
std::mutex g_scratch_mu;
std::vector<ScratchDev> g_scratch;  // by device ordinal

constexpr int64_t kImgAlign = 256;

int64_t img_align(int64_t b) { return (b + kImgAlign - 1) / kImgAlign * kImgAlign; }

}  // namespace

// Lay out the tables of `ex` and room for the records of one buffer set in
// ex->img; returns the image's size in bytes.
static int64_t build_image(const Plan& p, ExecState& ex) {
    const SliceTables t = slice_tables(ex);
    const int64_t sizes[8] = {
        int64_t(ex.htiles.size() * sizeof(int2)), int64_t(t.cuts.size() * sizeof(int64_t)),
        int64_t(t.soff.size() * sizeof(int32_t)), int64_t(t.sched.size() * sizeof(int32_t)),
        int64_t(t.tiles.size() * sizeof(int2)),   int64_t(t.runits.size() * sizeof(ResUnit)),
        int64_t(t.prog.size() * sizeof(uint32_t)),
        (ex.rec_words + p.n) * int64_t(sizeof(uint64_t))};
    int64_t at = 0;
    for (int i = 0; i < 8; ++i) {
        ex.img_off[i] = at;
        at = img_align(at + sizes[i]);
    }
    if (at > int64_t(AR_NOALLOC_MAX_BYTES)) return at;
    ex.img.assign(size_t(at / 8), 0);
    char* b = reinterpret_cast<char*>(ex.img.data());
    const void* src[7] = {ex.htiles.data(), t.cuts.data(), t.soff.data(), t.sched.data(),
                          t.tiles.data(), t.runits.data(), t.prog.data()};
    for (int i = 0; i < 7; ++i)
        if (sizes[i]) std::memcpy(b + ex.img_off[i], src[i], size_t(sizes[i]));
    return at;
}

AR_EXPORT ar_status ar_plan_execute_noalloc(ar_plan* plan, void* const* bufs, void* stream) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    if (!bufs) return fail(AR_ERR_INVALID_ARG, "bufs is NULL");
    try {
        if (plan->N == 0 || plan->num_phases() == 0) return AR_OK;
        ExecState* ex = exec_state(*plan);
        if (ex->launches.empty()) return AR_OK;
        const std::vector<void*> set(bufs, bufs + plan->n);
        ar_status s = check_buffers(*plan, set);
        if (s != AR_OK) return s;
        if (ex->img.empty()) {
            const int64_t need = build_image(*plan, *ex);
            if (ex->img.empty())
                return fail(AR_ERR_UNSUPPORTED,
                            "the plan's tables and step records take " + std::to_string(need) +
                                " bytes; ar_plan_execute_noalloc holds at most " +
                                std::to_string(int64_t(AR_NOALLOC_MAX_BYTES)));
        }
        int dev = -1;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("hipGetDevice", e));
        if (dev < 0) return fail(AR_ERR_HIP, "no current device");
        const hipStream_t st = static_cast<hipStream_t>(stream);
        uint8_t* base = nullptr;
        {
            std::lock_guard<std::mutex> lock(g_scratch_mu);
            if (size_t(dev) >= g_scratch.size()) g_scratch.resize(size_t(dev) + 1);
            ScratchDev& sd = g_scratch[size_t(dev)];
            if (!sd.ptr) {
                void* ptr = nullptr;
                e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
                if (e != hipSuccess || !ptr)
                    return fail(AR_ERR_HIP, hip_msg("hipGetSymbolAddress(scratch)", e));
                sd.ptr = static_cast<uint8_t*>(ptr);
            }
            base = sd.ptr;
            const bool tables = sd.serial != ex->serial;
            if (tables || sd.bufs != set) {
                const int64_t rec = ex->img_off[7];
                const int64_t end = int64_t(ex->img.size()) * 8;
                fill_records(*ex, bufs, plan->n,
                             ex->img.data() + rec / int64_t(sizeof(uint64_t)));
                const int64_t from = tables ? 0 : rec;
                sd.serial = 0;  // unknown until the copy is enqueued
                e = hipMemcpyAsync(base + from, reinterpret_cast<const char*>(ex->img.data()) + from,
                                   size_t(end - from), hipMemcpyHostToDevice, st);
                if (e != hipSuccess) return fail(AR_ERR_HIP, hip_msg("scratch upload", e));
                sd.serial = ex->serial;
                sd.bufs = set;
            }
        }
        auto at = [&](int i) { return base + ex->img_off[i]; };
        const DevView v{reinterpret_cast<const int2*>(at(0)), reinterpret_cast<const int64_t*>(at(1)),
                        reinterpret_cast<const int32_t*>(at(2)), reinterpret_cast<const int32_t*>(at(3)),
                        reinterpret_cast<const int2*>(at(4)), reinterpret_cast<const ResUnit*>(at(5)),
                        reinterpret_cast<const uint32_t*>(at(6)), reinterpret_cast<const uint64_t*>(at(7)),
                        buffers_aligned(bufs, plan->n)};
        return launch_all(plan, ex, v, st, nullptr);
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
    } else if (option == AR_OPT_RESIDENT) {
        if (value != 0 && value != 1) return fail(AR_ERR_INVALID_ARG, "AR_OPT_RESIDENT takes 0 or 1");
        field = &plan->resident;
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

AR_EXPORT ar_status ar_plan_launch_kernel(const ar_plan* plan, int32_t i, int32_t* kernel) {
    clear_error();
    if (!plan || !kernel) return fail(AR_ERR_INVALID_ARG, "NULL argument");
    try {
        const ExecState* ex = exec_state(const_cast<ar_plan&>(*plan));
        if (i < 0 || i >= int32_t(ex->stages.size()))
            return fail(AR_ERR_INVALID_ARG, "launch index out of range");
        const Stage stg = ex->stages[size_t(i)];
        if (stg.slice >= 0) {
            const SliceDesc& sd = ex->slices[size_t(stg.slice)];
            *kernel = sd.streamed ? AR_KERNEL_STREAM : sd.resident ? AR_KERNEL_RESIDENT
                                                                   : AR_KERNEL_SLICED;
        } else {
            *kernel = ex->launches[size_t(stg.launch)].dsplit > 1 ? AR_KERNEL_SPLIT
                                                                   : AR_KERNEL_PHASE;
        }
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
            if (phase) *phase = sd.streamed ? -3 : sd.resident ? -2 : -1;
            if (nsrc) *nsrc = sd.max_k;
            if (max_dst) *max_dst = sd.max_dst;
            if (num_steps) *num_steps = sd.nsteps;
            if (bytes) *bytes = sd.resident ? sd.res_bytes : sd.bytes;
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
