// Batched phase kernel for gfx950: one launch executes every step of one
// phase that has the same source count k (a copy is the k = 1 case); a step
// may store its result into several destinations.
//
// Work decomposition.  Each step's element range is cut into wave tiles of
// `tile_elems` elements, aligned to 16 bytes in the buffer; a 64-lane
// wavefront executes one tile.  A launch therefore covers all steps of the
// phase at once, whatever their number and length.  Tile -> (step, tile in
// step) is arithmetic when the steps are about equally long and otherwise
// comes from a per-launch table.
//
// Inner loop.  Per iteration every lane moves U 16-byte vectors of each of
// the K sources (global_load_dwordx4; the wave touches 1 KiB contiguous per
// vector slot), folds them in source order in fp32 (bf16 widened; int32 with
// wrap-around) and stores U vectors.  Loads are nontemporal unless the launch
// reads some range more than once, stores unless the launch's output is small
// enough to stay cached for the next phase.  Unaligned head and tail elements of a
// step are done element-wise.  A wave reads its step as one record with the
// buffer pointers already resolved (see StepHead): wave-uniform, in scalar
// registers after a single dependent load.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace arp {

enum DType : int32_t { DT_F32 = 0, DT_I32 = 1, DT_BF16 = 2 };

// One executed step: fold the k sources over [begin, end) and store the
// result into each of the ndst destinations.  Host form; the indices point
// into the plan's index pool, where a step's destinations that are not
// among its sources come first.
struct DevStep {
    int64_t begin;
    int64_t end;
    int32_t src_off;  // first source index in the index pool
    int32_t k;        // number of sources
    int32_t dst_off;  // first destination index in the same pool
    int32_t ndst;     // number of destinations
    int32_t nfree;    // the first nfree destinations are not sources of the step
};

// The record a kernel reads for a step, built per buffer set: this header
// (4 words) followed by k source and ndst destination buffer pointers, one
// 8-byte word each, the nfree destinations that are not sources first.
// Records of one launch have a common stride, so a wave finds its step's
// pointers with one dependent load.
struct StepHead {
    int64_t begin;
    int64_t end;
    int32_t k;
    int32_t ndst;
    int32_t nfree;
    int32_t pad;
};
constexpr int kRecHead = 4;  // header words

// Per source count K (K = 0: source count read at run time):
//   U   16-byte vectors in flight per lane and source,
//   WPB wavefronts per block,
//   TE  largest wave tile, in 16-byte vectors per source.
// Chosen by measurement on MI355X: a 2-input fold and a copy stream best
// with 16 KiB per source per wave and 8-wave blocks; wide folds want fewer
// vectors per source in flight and smaller tiles.  The 16-source fold runs
// best with one 1 KiB vector slot per source and tile (6.06 TB/s on 1 GiB,
// against 5.86 with 4 KiB tiles; 2 slots per lane, 512-vector tiles or
// 8-wave blocks were slower still).
struct KCfg {
    int U, WPB, TE;
};
constexpr int kWideU = 16;   // vectors per lane and source of the wide 2-source pass
constexpr int kWideU8 = 4;   // ... and of the wide 8-source pass (4-byte elements)
__host__ __device__ constexpr KCfg kcfg(int K) {
    return K == 1 ? KCfg{16, 8, 1024}
         : K == 2 ? KCfg{8, 8, 1024}
         : K <= 4 && K > 0 ? KCfg{4, 4, 512}
         : K == 8 ? KCfg{2, 4, 256}
         : K == 16 ? KCfg{1, 4, 64}
         : KCfg{4, 4, 256};
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Buffer pointers come from a table of generic pointers; marking them as
// global-memory pointers lets the compiler use global_load/global_store
// (vector memory counter only) instead of flat instructions.
#define AR_GLOBAL __attribute__((address_space(1)))
typedef AR_GLOBAL u32x4 gvec;
#define AR_LDS __attribute__((address_space(3)))

template <class T>
__device__ __forceinline__ AR_GLOBAL T* as_global(void* p) {
    return (AR_GLOBAL T*)(p);
}

// Vector loads and stores; NT marks them nontemporal (data that will not be
// touched again soon streams past the caches).
template <bool NT>
__device__ __forceinline__ u32x4 vload(const gvec* p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    else return *p;
}
template <bool NT>
__device__ __forceinline__ void vstore(gvec* p, u32x4 v) {
    if constexpr (NT) __builtin_nontemporal_store(v, p);
    else *p = v;
}

template <int DT> struct Elem;
template <> struct Elem<DT_F32> { using T = float;    static constexpr int VEC = 4; };
template <> struct Elem<DT_I32> { using T = uint32_t; static constexpr int VEC = 4; };
template <> struct Elem<DT_BF16> { using T = uint16_t; static constexpr int VEC = 8; };

// ---------------------------------------------------------------- bf16

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// fp32 -> bf16, round to nearest, ties to even; a NaN keeps its sign and
// upper payload bits and gets the quiet bit.  gfx950 does this in hardware,
// two values per instruction (v_cvt_pk_bf16_f32), denormals included when
// fp32 denormals are enabled (they are: -fno-gpu-flush-denormals-to-zero).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t bf16_pack(float lo, float hi) {
    const f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// ---------------------------------------------- 16-byte vector accumulator

template <int DT> struct VAcc;

template <> struct VAcc<DT_F32> {
    float v[4];
    __device__ __forceinline__ void init(const u32x4 x) {
        v[0] = __uint_as_float(x[0]); v[1] = __uint_as_float(x[1]);
        v[2] = __uint_as_float(x[2]); v[3] = __uint_as_float(x[3]);
    }
    __device__ __forceinline__ void add(const u32x4 x) {
        v[0] += __uint_as_float(x[0]); v[1] += __uint_as_float(x[1]);
        v[2] += __uint_as_float(x[2]); v[3] += __uint_as_float(x[3]);
    }
    __device__ __forceinline__ u32x4 out() const {
        return u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]),
                     __float_as_uint(v[2]), __float_as_uint(v[3])};
    }
};

template <> struct VAcc<DT_I32> {
    uint32_t v[4];
    __device__ __forceinline__ void init(const u32x4 x) { v[0] = x[0]; v[1] = x[1]; v[2] = x[2]; v[3] = x[3]; }
    __device__ __forceinline__ void add(const u32x4 x) { v[0] += x[0]; v[1] += x[1]; v[2] += x[2]; v[3] += x[3]; }
    __device__ __forceinline__ u32x4 out() const { return u32x4{v[0], v[1], v[2], v[3]}; }
};

template <> struct VAcc<DT_BF16> {
    float v[8];
    __device__ __forceinline__ void init(const u32x4 x) {
        v[0] = bf16_lo(x[0]); v[1] = bf16_hi(x[0]); v[2] = bf16_lo(x[1]); v[3] = bf16_hi(x[1]);
        v[4] = bf16_lo(x[2]); v[5] = bf16_hi(x[2]); v[6] = bf16_lo(x[3]); v[7] = bf16_hi(x[3]);
    }
    __device__ __forceinline__ void add(const u32x4 x) {
        v[0] += bf16_lo(x[0]); v[1] += bf16_hi(x[0]); v[2] += bf16_lo(x[1]); v[3] += bf16_hi(x[1]);
        v[4] += bf16_lo(x[2]); v[5] += bf16_hi(x[2]); v[6] += bf16_lo(x[3]); v[7] += bf16_hi(x[3]);
    }
    __device__ __forceinline__ u32x4 out() const {
        return u32x4{bf16_pack(v[0], v[1]), bf16_pack(v[2], v[3]),
                     bf16_pack(v[4], v[5]), bf16_pack(v[6], v[7])};
    }
};

// ------------------------------------------------ single-element accumulator

template <int DT> struct SAcc;
template <> struct SAcc<DT_F32> {
    float v;
    __device__ __forceinline__ void init(float x) { v = x; }
    __device__ __forceinline__ void add(float x) { v += x; }
    __device__ __forceinline__ float out() const { return v; }
};
template <> struct SAcc<DT_I32> {
    uint32_t v;
    __device__ __forceinline__ void init(uint32_t x) { v = x; }
    __device__ __forceinline__ void add(uint32_t x) { v += x; }
    __device__ __forceinline__ uint32_t out() const { return v; }
};
template <> struct SAcc<DT_BF16> {
    float v;
    __device__ __forceinline__ void init(uint16_t x) { v = __uint_as_float(uint32_t(x) << 16); }
    __device__ __forceinline__ void add(uint16_t x) { v += __uint_as_float(uint32_t(x) << 16); }
    __device__ __forceinline__ uint16_t out() const { return uint16_t(bf16_pack(v, 0.0f)); }
};

// Element ranges of wave tile t of a step [begin, end): the tile is
// [lo, hi); inside it [vlo, vhi) is done with 16-byte vectors and the head
// [lo, vlo) and tail [vhi, hi) element-wise.  Tiles are aligned to 16 bytes
// of the buffer (`vecok`: every buffer base is 16-byte aligned), so only the
// first and last tile of a step have a head or tail.  Shared by the kernel
// and the host-side tiling check.
struct TileSpan {
    int64_t lo, hi, vlo, vhi;
};

__host__ __device__ __forceinline__ TileSpan tile_span(int64_t begin, int64_t end,
                                                       int64_t t, int64_t te,
                                                       int64_t vec, bool vecok) {
    TileSpan r;
    const int64_t abase = vecok ? (begin & ~(vec - 1)) : begin;
    const int64_t a = abase + t * te, b = abase + (t + 1) * te;
    r.lo = a > begin ? a : begin;
    r.hi = b < end ? b : end;
    r.vlo = r.vhi = r.hi;
    if (vecok && r.lo < r.hi) {
        const int64_t vlo = (r.lo + vec - 1) & ~(vec - 1);
        const int64_t vhi = r.hi & ~(vec - 1);
        if (vhi > vlo) {
            r.vlo = vlo;
            r.vhi = vhi;
        }
    }
    return r;
}

// Wave tile `unit` of a launch -> (step s within the launch, tile t of it):
// from the launch's tile table when it has one, else arithmetic with a
// fixed number of tiles per step.
__host__ __device__ __forceinline__ void unit_tile(int64_t unit, const int2* tiles,
                                                   int64_t tiles_per_step,
                                                   int64_t& s, int64_t& t) {
    if (tiles) {
        const int2 e = tiles[unit];
        s = e.x;
        t = e.y;
    } else {
        s = unit / tiles_per_step;
        t = unit - s * tiles_per_step;
    }
}

__device__ __forceinline__ int64_t uniform64(int64_t x) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(uint64_t(x)));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(uint64_t(x) >> 32));
    return int64_t((uint64_t(hi) << 32) | lo);
}

// Fold elements [lo, hi) of the k sources sp[] into the destinations dp[],
// one element per lane per pass (used for unaligned heads/tails and for
// unaligned buffers).
template <int DT, int K>
__device__ __forceinline__ void fold_scalar(void* const* __restrict__ sp, int k,
                                            void* const* __restrict__ dp, int ndst,
                                            int64_t lo, int64_t hi, int lane) {
    using T = typename Elem<DT>::T;
    if (K == 1 || (K == 0 && k == 1)) {  // copy: move the bits unchanged
        const AR_GLOBAL T* s = as_global<T>(sp[0]);
        for (int64_t e = lo + lane; e < hi; e += 64) {
            const T v = s[e];
            for (int j = 0; j < ndst; ++j) as_global<T>(dp[j])[e] = v;
        }
        return;
    }
    constexpr int SU = 4;
    for (int64_t e0 = lo; e0 < hi; e0 += 64 * SU) {
        SAcc<DT> acc[SU];
        bool ok[SU];
#pragma unroll
        for (int u = 0; u < SU; ++u) ok[u] = e0 + u * 64 + lane < hi;
        {
            const AR_GLOBAL T* s = as_global<T>(sp[0]);
#pragma unroll
            for (int u = 0; u < SU; ++u)
                if (ok[u]) acc[u].init(s[e0 + u * 64 + lane]);
        }
        const int kk = K ? K : k;
        for (int t = 1; t < kk; ++t) {
            const AR_GLOBAL T* s = as_global<T>(sp[t]);
#pragma unroll
            for (int u = 0; u < SU; ++u)
                if (ok[u]) acc[u].add(s[e0 + u * 64 + lane]);
        }
        for (int j = 0; j < ndst; ++j) {
            AR_GLOBAL T* d = as_global<T>(dp[j]);
#pragma unroll
            for (int u = 0; u < SU; ++u)
                if (ok[u]) d[e0 + u * 64 + lane] = acc[u].out();
        }
    }
}

// Destination pointers of a step, two ways.  Dsts holds the first kRegDst
// in registers for a whole tile (read once: re-reading them from the record
// after every store would cost a dependent load per iteration, since the
// compiler cannot tell the stores from the record) and reads the rest from
// the record; the phase kernel, which loops over a tile, uses it.  DstMem
// reads them from the record at the store; the sliced kernel, which stores
// each step once, uses it.
constexpr int kRegDst = 8;
struct Dsts {
    void* r[kRegDst];
    void* const* more;  // destinations kRegDst.. (in the record)
    int n;
};
struct DstMem {
    void* const* p;
    int n;
};
__device__ __forceinline__ Dsts load_dsts(void* const* __restrict__ dp, int ndst) {
    Dsts d;
#pragma unroll
    for (int j = 0; j < kRegDst; ++j) d.r[j] = j < ndst ? dp[j] : nullptr;
    d.more = dp + kRegDst;
    d.n = ndst;
    return d;
}

// Store U vectors per lane (vector offset `at` + u * 64 + lane) into each
// destination; every load of these positions happened before, so a
// destination may also be one of the sources.
template <int U, int CM, bool FULL>
__device__ __forceinline__ void store_all(const Dsts& dst, int64_t v0, const u32x4 (&out)[U],
                                          const bool (&ok)[U], int64_t at, int lane) {
#pragma unroll
    for (int j = 0; j < kRegDst; ++j) {
        if (j < dst.n) {
            gvec* d = as_global<u32x4>(dst.r[j]) + v0 + at + lane;
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (FULL || ok[u]) vstore<(CM & 2) != 0>(d + u * 64, out[u]);
        }
    }
    for (int j = kRegDst; j < dst.n; ++j) {
        gvec* d = as_global<u32x4>(dst.more[j - kRegDst]) + v0 + at + lane;
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (FULL || ok[u]) vstore<(CM & 2) != 0>(d + u * 64, out[u]);
    }
}
template <int U, int CM, bool FULL>
__device__ __forceinline__ void store_all(const DstMem& dst, int64_t v0, const u32x4 (&out)[U],
                                          const bool (&ok)[U], int64_t at, int lane) {
    for (int j = 0; j < dst.n; ++j) {
        gvec* d = as_global<u32x4>(dst.p[j]) + v0 + at + lane;
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (FULL || ok[u]) vstore<(CM & 2) != 0>(d + u * 64, out[u]);
    }
}

// The loads and adds of fold_vectors (below) without its stores, for split
// tiles, which store in two parts around a barrier (split_pass): out[u] is
// the folded vector u, ok[u] whether it is in range.  fold_vectors keeps its
// own copy of these lines: built on this function, its loop compiled to a
// different schedule and the 3 GiB two-source fold ran 3 % slower.
template <int DT, int K, int U, int CM, bool FULL>
__device__ __forceinline__ void fold_load(const gvec* const* sp, int64_t at, int64_t nv,
                                          int lane, u32x4 (&out)[U], bool (&ok)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) ok[u] = FULL || at + u * 64 + lane < nv;
    u32x4 x[K][U];
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) x[j][u] = vload<(CM & 1) != 0>(sp[j] + at + u * 64 + lane);
    if constexpr (K == 1) {
#pragma unroll
        for (int u = 0; u < U; ++u) out[u] = x[0][u];
    } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            VAcc<DT> acc;
            acc.init(x[0][u]);
#pragma unroll
            for (int j = 1; j < K; ++j) acc.add(x[j][u]);
            out[u] = acc.out();
        }
    }
}
// U vectors per lane of K sources at vector offset `at` (+ u * 64 + lane),
// folded in source order and stored to every destination.  FULL: all U
// vectors are in range, so the loads are issued back to back with no
// per-vector branch.  Cache mode CM of a launch: bit 0 = nontemporal loads,
// bit 1 = nontemporal stores.
template <int DT, int K, int U, int CM, bool FULL, class D>
__device__ __forceinline__ void fold_vectors(const gvec* const* sp, const D& dst,
                                             int64_t v0, int64_t at, int64_t nv, int lane) {
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) ok[u] = FULL || at + u * 64 + lane < nv;
    u32x4 x[K][U];
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) x[j][u] = vload<(CM & 1) != 0>(sp[j] + at + u * 64 + lane);
    u32x4 out[U];
    if constexpr (K == 1) {
#pragma unroll
        for (int u = 0; u < U; ++u) out[u] = x[0][u];
    } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            VAcc<DT> acc;
            acc.init(x[0][u]);
#pragma unroll
            for (int j = 1; j < K; ++j) acc.add(x[j][u]);
            out[u] = acc.out();
        }
    }
    store_all<U, CM, FULL>(dst, v0, out, ok, at, lane);
}

// Runtime source count: the sources in groups of `group` (1..kRtGroup),
// every load of a group in flight at once (U vectors per lane and source),
// then added in source order, so the fold is the same left fold as the
// unrolled kernels'.  Short launches want the loads of several sources in
// flight; long ones stream best one source at a time (more loads per wave
// cost occupancy where there is work enough to hide the latency).
constexpr int kRtGroup = 4;

// fold_load for a runtime source count (as fold_vectors_rt, below, without
// its stores).
template <int DT, int U, int CM, bool FULL>
__device__ __forceinline__ void fold_load_rt(void* const* __restrict__ srcp, int k, int64_t v0,
                                             int64_t at, int64_t nv, int lane, int group,
                                             u32x4 (&out)[U], bool (&ok)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) ok[u] = FULL || at + u * 64 + lane < nv;
    if (k == 1) {
        const gvec* s0 = as_global<u32x4>(srcp[0]) + v0;
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) out[u] = vload<(CM & 1) != 0>(s0 + at + u * 64 + lane);
    } else {
        VAcc<DT> acc[U];
        for (int j0 = 0; j0 < k; j0 += group) {
            u32x4 x[kRtGroup][U];
#pragma unroll
            for (int g = 0; g < kRtGroup; ++g) {
                if (g < group && j0 + g < k) {  // wave-uniform
                    const gvec* sj = as_global<u32x4>(srcp[j0 + g]) + v0;
#pragma unroll
                    for (int u = 0; u < U; ++u)
                        if (ok[u]) x[g][u] = vload<(CM & 1) != 0>(sj + at + u * 64 + lane);
                }
            }
#pragma unroll
            for (int g = 0; g < kRtGroup; ++g) {
                if (g < group && j0 + g < k) {
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        if (j0 + g == 0) acc[u].init(x[g][u]);
                        else acc[u].add(x[g][u]);
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) out[u] = acc[u].out();
    }
}
template <int DT, int U, int CM, bool FULL, class D>
__device__ __forceinline__ void fold_vectors_rt(void* const* __restrict__ srcp, int k,
                                                const D& dst, int64_t v0, int64_t at,
                                                int64_t nv, int lane, int group) {
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) ok[u] = FULL || at + u * 64 + lane < nv;
    u32x4 out[U];
    if (k == 1) {
        const gvec* s0 = as_global<u32x4>(srcp[0]) + v0;
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) out[u] = vload<(CM & 1) != 0>(s0 + at + u * 64 + lane);
    } else {
        VAcc<DT> acc[U];
        for (int j0 = 0; j0 < k; j0 += group) {
            u32x4 x[kRtGroup][U];
#pragma unroll
            for (int g = 0; g < kRtGroup; ++g) {
                if (g < group && j0 + g < k) {  // wave-uniform
                    const gvec* sj = as_global<u32x4>(srcp[j0 + g]) + v0;
#pragma unroll
                    for (int u = 0; u < U; ++u)
                        if (ok[u]) x[g][u] = vload<(CM & 1) != 0>(sj + at + u * 64 + lane);
                }
            }
#pragma unroll
            for (int g = 0; g < kRtGroup; ++g) {
                if (g < group && j0 + g < k) {
#pragma unroll
                    for (int u = 0; u < U; ++u) {
                        if (j0 + g == 0) acc[u].init(x[g][u]);
                        else acc[u].add(x[g][u]);
                    }
                }
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) out[u] = acc[u].out();
    }
    store_all<U, CM, FULL>(dst, v0, out, ok, at, lane);
}

// Split launches.  A wave storing one small tile to many destinations
// spends its time issuing the stores (measured on MI355X: 512 waves each
// storing 1 KiB to 64 buffers take 13.5 us, 2048 waves storing 16 each
// 7.4 us).  A launch of few tiles whose steps have many destinations
// therefore gives each tile a whole workgroup (dsplit = wavefronts per
// block): every wave folds the tile and stores to its share of the
// destinations.  The destinations that are sources of the step as well
// (they come last in the record) are stored only after a workgroup barrier,
// when every wave has loaded the sources; the others are stored at once.
// This pays only where each tile runs on the XCD that wrote its sources in
// the launch before (the host places tiles so): the bf16 tree (8, 8, 8)'s
// level-2 reduce into 64 buffers takes 12.5 us so, 26 us split with tiles on
// other XCDs, 20 us unsplit.
// kSplitWaves: wavefronts per workgroup (and tile) of a split launch.
// split_share: part `part` of `parts` gets items [a, b) of n, contiguous,
// the shares differing by at most one.  Shared with the host-side check.
constexpr int kSplitWaves = 4;
__host__ __device__ __forceinline__ void split_share(int n, int part, int parts, int& a, int& b) {
    const int q = n / parts, r = n % parts;
    a = part * q + (part < r ? part : r);
    b = a + q + (part < r ? 1 : 0);
}

// One pass of a split tile: fold U vectors per lane at `at`, store them to
// this wave's share of the destinations that are not sources (fd), and,
// when the step has destinations among its sources, wait for the
// workgroup and store to this wave's share of those (sd).
template <int DT, int K, int U, int CM, bool FULL>
__device__ __forceinline__ void split_pass(const gvec* const* sv, void* const* __restrict__ sp,
                                           int k, int rt_group, const Dsts& fd, const DstMem& sd,
                                           bool sync, int64_t v0, int64_t at, int64_t nv,
                                           int lane) {
    u32x4 out[U];
    bool ok[U];
    if constexpr (K > 0) fold_load<DT, K, U, CM, FULL>(sv, at, nv, lane, out, ok);
    else fold_load_rt<DT, U, CM, FULL>(sp, k, v0, at, nv, lane, rt_group, out, ok);
    store_all<U, CM, FULL>(fd, v0, out, ok, at, lane);
    if (sync) {
        __syncthreads();
        store_all<U, CM, FULL>(sd, v0, out, ok, at, lane);
    }
}

// A tile run by the `parts` waves of a workgroup, this one being `part`
// (buffers 16-byte aligned).  Every wave takes the same branches and passes
// (same step and tile), so all reach the same barriers.  Element-wise heads
// and tails are done by the first wave alone, with every destination: no
// other wave touches those positions.
template <int DT, int K, int CM>
__device__ __forceinline__ void split_tile(void* const* __restrict__ sp, int k,
                                           void* const* __restrict__ dp, int ndst, int nfree,
                                           const TileSpan& ts, int part, int parts, int lane,
                                           int rt_group) {
    constexpr int VEC = Elem<DT>::VEC;
    constexpr int U = kcfg(K).U;
    if (part == 0) {
        if (ts.vlo > ts.lo) fold_scalar<DT, K>(sp, k, dp, ndst, ts.lo, ts.vlo, lane);
        if (ts.hi > ts.vhi) fold_scalar<DT, K>(sp, k, dp, ndst, ts.vhi, ts.hi, lane);
    }
    if (ts.vhi <= ts.vlo) return;
    const int64_t v0 = ts.vlo / VEC;
    const int64_t nv = (ts.vhi - ts.vlo) / VEC;
    int f0, f1, g0, g1;
    split_share(nfree, part, parts, f0, f1);
    split_share(ndst - nfree, part, parts, g0, g1);
    const Dsts fd = load_dsts(dp + f0, f1 - f0);
    const DstMem sd{dp + nfree + g0, g1 - g0};
    const bool sync = ndst > nfree;
    const gvec* sv[K > 0 ? K : 1];
    if constexpr (K > 0) {
#pragma unroll
        for (int j = 0; j < K; ++j) sv[j] = as_global<u32x4>(sp[j]) + v0;
    }
    int64_t at = 0;
    for (; at + 64 * U <= nv; at += 64 * U)
        split_pass<DT, K, U, CM, true>(sv, sp, k, rt_group, fd, sd, sync, v0, at, nv, lane);
    if (at < nv)
        split_pass<DT, K, U, CM, false>(sv, sp, k, rt_group, fd, sd, sync, v0, at, nv, lane);
}

// One launch: `nunits` wave tiles over the steps whose records start at
// `recs`, `stride` words apart.  K = 0 means the source count is read from
// each step (any k >= 1), folded `rt_group` sources at a time.  VECOK: every
// buffer is 16-byte aligned.  CM: cache mode of the vector loads and stores.
// UW (0: kcfg's U) overrides the vectors per lane and source of a pass: the
// wide 2-source instance (kWideU) loads a whole 1024-vector tile in one pass,
// so no load of a tile waits behind one of its stores (the two share the
// wave's in-order memory counter); it pays on multi-GiB launches with
// nontemporal loads and stores (RHD's first halving launch, 3 GiB: 531 ->
// 520 us), while its 148 VGPRs (3 waves per SIMD, against 5) made short
// launches slower (bf16 Ring as written +10-15 %).  The wide 8-source
// instance (kWideU8, 4-byte elements) likewise covers its 256-vector tile in
// one pass instead of two.
template <int DT, int K, bool VECOK, int CM, int UW = 0>
__global__ __launch_bounds__(64 * kcfg(K).WPB) void phase_kernel(
    const uint64_t* __restrict__ recs, int64_t stride, const int2* __restrict__ tiles,
    int64_t nunits, int64_t tiles_per_step, int64_t tile_elems, int rt_group) {
    constexpr int VEC = Elem<DT>::VEC;
    constexpr int U = UW ? UW : kcfg(K).U;
    constexpr int WPB = kcfg(K).WPB;
    const int lane = int(threadIdx.x) & 63;
    const int64_t unit = int64_t(blockIdx.x) * WPB +
                         int64_t(__builtin_amdgcn_readfirstlane(threadIdx.x >> 6));
    if (unit >= nunits) return;
    int64_t s, t;
    unit_tile(unit, tiles, tiles_per_step, s, t);
    s = uniform64(s);
    t = uniform64(t);
    if (s < 0) return;  // a padding entry of a tile table
    const uint64_t* rec = recs + s * stride;
    const StepHead st = *reinterpret_cast<const StepHead*>(rec);
    const int k = K ? K : st.k;
    void* const* sp = reinterpret_cast<void* const*>(rec + kRecHead);
    void* const* dp = sp + k;
    const int ndst = st.ndst;

    const TileSpan ts = tile_span(st.begin, st.end, t, tile_elems, VEC, VECOK);
    if (ts.lo >= ts.hi) return;
    if (ts.vlo > ts.lo) fold_scalar<DT, K>(sp, k, dp, ndst, ts.lo, ts.vlo, lane);
    if (ts.hi > ts.vhi) fold_scalar<DT, K>(sp, k, dp, ndst, ts.vhi, ts.hi, lane);
    if (!VECOK || ts.vhi <= ts.vlo) return;

    const int64_t v0 = ts.vlo / VEC;
    const int64_t nv = (ts.vhi - ts.vlo) / VEC;
    const Dsts dst = load_dsts(dp, ndst);
    int64_t at = 0;
    if constexpr (K > 0) {
        const gvec* sv[K];
#pragma unroll
        for (int j = 0; j < K; ++j) sv[j] = as_global<u32x4>(sp[j]) + v0;
        for (; at + 64 * U <= nv; at += 64 * U)
            fold_vectors<DT, K, U, CM, true>(sv, dst, v0, at, nv, lane);
        if (at < nv) fold_vectors<DT, K, U, CM, false>(sv, dst, v0, at, nv, lane);
    } else {
        for (; at + 64 * U <= nv; at += 64 * U)
            fold_vectors_rt<DT, U, CM, true>(sp, k, dst, v0, at, nv, lane, rt_group);
        if (at < nv)
            fold_vectors_rt<DT, U, CM, false>(sp, k, dst, v0, at, nv, lane, rt_group);
    }
}

// Split launch (see split_tile): workgroup b runs wave tile b of the
// launch's tile table (tiles[b] = (step, tile in step), or (-1, 0) padding),
// its kSplitWaves waves each storing to a share of the destinations.
// Buffers are 16-byte aligned (a split launch on unaligned buffers runs
// phase_kernel over the same table instead).  CM: cache mode of the vector
// stores (bit 1); the loads are cached, since every wave of the workgroup
// reads the sources.
// A kernel of its own, so that phase_kernel's code stays as it was: with
// the split path inside it, the compiler scheduled the fold loop's loads
// and stores differently and the 3 GiB two-source fold ran 3 % slower.
template <int DT, int K, int CM>
__global__ __launch_bounds__(64 * kSplitWaves) void split_kernel(
    const uint64_t* __restrict__ recs, int64_t stride, const int2* __restrict__ tiles,
    int64_t ntiles, int64_t tile_elems, int rt_group) {
    constexpr int VEC = Elem<DT>::VEC;
    const int lane = int(threadIdx.x) & 63;
    const int part = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
    const int64_t tile = blockIdx.x;
    if (tile >= ntiles) return;
    const int2 e = tiles[tile];
    const int64_t s = __builtin_amdgcn_readfirstlane(e.x);
    const int64_t t = __builtin_amdgcn_readfirstlane(e.y);
    if (s < 0) return;  // a padding entry of the table
    const uint64_t* rec = recs + s * stride;
    const StepHead st = *reinterpret_cast<const StepHead*>(rec);
    const int k = K ? K : st.k;
    void* const* sp = reinterpret_cast<void* const*>(rec + kRecHead);
    const TileSpan ts = tile_span(st.begin, st.end, t, tile_elems, VEC, true);
    if (ts.lo >= ts.hi) return;
    split_tile<DT, K, CM>(sp, k, sp + k, st.ndst, st.nfree, ts, part, kSplitWaves, lane,
                          rt_group);
}

// ------------------------------------------------------------------------
// Sliced kernel: one launch for a run of consecutive phases whose launches
// would be too short to fill the chip.
//
// Every step is element-wise and the steps of a phase are independent, so
// the value at an element position depends only on what earlier phases did
// at that same position.  Here each wavefront owns a fixed tile of element
// positions (inside one segment: the element ranges between consecutive
// step boundaries of the run) and carries it through the run's phases in
// order: in phase p it runs, for its tile, every step of p that covers the
// segment, reading and writing the buffers in memory exactly as the
// phase-by-phase execution does.  A lane always handles the same positions,
// so it only ever reads back what it wrote itself: no barrier between
// phases, one launch for the run.
constexpr int kSliceU = 4;    // vectors per lane in a tile
constexpr int kSliceWPB = 4;  // wavefronts per block

template <int DT, int K>
__device__ __forceinline__ void slice_fold(void* const* __restrict__ sp,
                                           void* const* __restrict__ dp, int ndst,
                                           int64_t v0, int64_t nv, int lane) {
    const gvec* sv[K];
#pragma unroll
    for (int j = 0; j < K; ++j) sv[j] = as_global<u32x4>(sp[j]) + v0;
    const DstMem dst{dp, ndst};
    if (nv == 64 * kSliceU)
        fold_vectors<DT, K, kSliceU, 0, true>(sv, dst, v0, 0, nv, lane);
    else
        fold_vectors<DT, K, kSliceU, 0, false>(sv, dst, v0, 0, nv, lane);
}

// sched lists, per (phase of the slice, segment), the word offsets in
// `recs` of the records of the steps covering the segment.
template <int DT>
__global__ __launch_bounds__(64 * kSliceWPB) void sliced_kernel(
    const uint64_t* __restrict__ recs, const int32_t* __restrict__ sched_off,
    const int32_t* __restrict__ sched, const int64_t* __restrict__ cuts,
    const int2* __restrict__ tiles, int64_t nunits, int32_t nphases, int32_t nseg,
    int64_t tile_elems) {
    constexpr int VEC = Elem<DT>::VEC;
    const int lane = int(threadIdx.x) & 63;
    const int64_t unit = int64_t(blockIdx.x) * kSliceWPB +
                         int64_t(__builtin_amdgcn_readfirstlane(threadIdx.x >> 6));
    if (unit >= nunits) return;
    const int2 e = tiles[unit];
    const int32_t seg = __builtin_amdgcn_readfirstlane(e.x);
    const int64_t t = __builtin_amdgcn_readfirstlane(e.y);
    const int64_t lo = cuts[seg] + t * tile_elems;
    const int64_t hi = min(cuts[seg + 1], lo + tile_elems);
    const int64_t v0 = lo / VEC;
    const int64_t nv = (hi - lo) / VEC;
    for (int32_t p = 0; p < nphases; ++p) {
        const int32_t a = sched_off[int64_t(p) * nseg + seg];
        const int32_t b = sched_off[int64_t(p) * nseg + seg + 1];
        for (int32_t i = a; i < b; ++i) {
            const uint64_t* rec = recs + sched[i];
            const StepHead st = *reinterpret_cast<const StepHead*>(rec);
            void* const* sp = reinterpret_cast<void* const*>(rec + kRecHead);
            void* const* dp = sp + st.k;
            switch (st.k) {
                case 1: slice_fold<DT, 1>(sp, dp, st.ndst, v0, nv, lane); break;
                case 2: slice_fold<DT, 2>(sp, dp, st.ndst, v0, nv, lane); break;
                case 4: slice_fold<DT, 4>(sp, dp, st.ndst, v0, nv, lane); break;
                case 8: slice_fold<DT, 8>(sp, dp, st.ndst, v0, nv, lane); break;
                default: {
                    const DstMem dst{dp, st.ndst};
                    if (nv == 64 * kSliceU)
                        fold_vectors_rt<DT, kSliceU, 0, true>(sp, st.k, dst, v0, 0, nv, lane,
                                                              kRtGroup);
                    else
                        fold_vectors_rt<DT, kSliceU, 0, false>(sp, st.k, dst, v0, 0, nv, lane,
                                                               kRtGroup);
                }
            }
        }
    }
}

}  // namespace arp
