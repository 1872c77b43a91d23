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
            std::vector<ResUnit> runits;
            std::vector<uint32_t> prog;
            for (const SliceDesc& sd : ex.slices) {
                cuts.insert(cuts.end(), sd.cuts.begin(), sd.cuts.end());
                soff.insert(soff.end(), sd.sched_off.begin(), sd.sched_off.end());
                sched.insert(sched.end(), sd.sched.begin(), sd.sched.end());
                tiles.insert(tiles.end(), sd.tiles.begin(), sd.tiles.end());
                runits.insert(runits.end(), sd.runits.begin(), sd.runits.end());
                prog.insert(prog.end(), sd.prog.begin(), sd.prog.end());
            }
            s = upload(&d->cuts, cuts, "segment table");
            if (s == AR_OK) s = upload(&d->sched_off, soff, "schedule offsets");
            if (s == AR_OK) s = upload(&d->sched, sched, "schedule");
            if (s == AR_OK) s = upload(&d->stiles, tiles, "slice tiles");
            if (s == AR_OK) s = upload(&d->runits, runits, "resident units");
            if (s == AR_OK) s = upload(&d->prog, prog, "resident programs");
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
    for (size_t i = 0; i < bufs.size(); ++i) w[ex.rec_words + int64_t(i)] = reinterpret_cast<uint64_t>(bufs[i]);
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
            if (stg.slice >= 0 && ex->slices[size_t(stg.slice)].resident) {
                const SliceDesc& sd = ex->slices[size_t(stg.slice)];
                const dim3 grid(static_cast<uint32_t>(sd.nunits)), block(64 * sd.res_waves);
                const size_t lds = size_t(plan->n) * 1024;
#define AR_RESIDENT(DT, W)                                                                    \
    hipLaunchKernelGGL((resident_kernel<DT, W>), grid, block, lds, stream, pe->dev + ex->rec_words, \
                       plan->n, d->runits + sd.runit_base, d->prog + sd.prog_base, sd.nunits)
                const bool four = sd.res_waves == 4;
                switch (plan->dtype) {
                    case AR_F32: if (four) AR_RESIDENT(DT_F32, 4); else AR_RESIDENT(DT_F32, 1); break;
                    case AR_I32: if (four) AR_RESIDENT(DT_I32, 4); else AR_RESIDENT(DT_I32, 1); break;
                    default: if (four) AR_RESIDENT(DT_BF16, 4); else AR_RESIDENT(DT_BF16, 1); break;
                }
#undef AR_RESIDENT
            } else if (stg.slice >= 0) {
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
            if (sd.resident) {
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
                    int32_t nw = -1;
                    for (int64_t i = 0; i < sd.nunits; ++i)
                        if (sd.tiles[size_t(i)].x == sg) {
                            nw = sd.runits[size_t(i)].nw;
                            break;
                        }
                    if (off < 0 || nw < 1 || int64_t(off) + nw > int64_t(sd.prog.size()))
                        return bad("resident records outside the table");
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
                            if (have[b] != want[b]) return bad("resident result differs from the phases' steps");
                        } else if (want[b] != input[b]) {
                            return bad("resident launch leaves a written row unstored");
                        }
                    }
                    words[size_t(sg)] = nw;
                }
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
        if (units)
            for (size_t i = 0; i < sd.runits.size(); ++i) {
                const ResUnit& u = sd.runits[i];
                int64_t* o = units + 6 * i;
                o[0] = u.lo;
                o[1] = int64_t(u.load);
                o[2] = int64_t(u.store);
                o[3] = u.nv;
                o[4] = u.off;
                o[5] = u.nw;
            }
        if (prog) std::copy(sd.prog.begin(), sd.prog.end(), prog);
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
            if (phase) *phase = sd.resident ? -2 : -1;
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
