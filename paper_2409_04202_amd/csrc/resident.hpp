// Resident sliced kernel for gfx950 (see below); it shares the vector
// types and the fold arithmetic of the phase and sliced kernels.
#pragma once

#include "kernels.hpp"

namespace arp {

// ------------------------------------------------------------------------
// Resident sliced kernel: the same runs of phases, with the element
// positions a workgroup owns kept on chip for the whole run.  A workgroup
// owns up to one 16-byte vector per lane inside one segment and holds it,
// for every buffer, in a 1 KiB LDS row (row b, lane l at rows[b * 64 + l]).
// Its W wavefronts (1 or 4) load the rows the run reads before writing them
// (global_load_lds_dwordx4: straight into LDS, all in flight at once; wave w
// takes the rows b with b % W == w), run the steps of every phase of the run
// on the rows (with four waves each wave on its own quarter of every row,
// ResLane), and store the rows the run wrote.  NT marks the row loads and
// stores nontemporal (cache policy NT), for runs whose traffic is larger
// than the last-level cache.  Four waves issue the row loads and stores and
// run the steps four times as fast; one wave per workgroup lets a compute
// unit hold more tiles when LDS does not limit it.
// A phase costs a few LDS accesses instead of a round trip through the
// memory hierarchy, and each buffer position is read and written once per
// run.
//
// Each workgroup reads one ResUnit: its tile, the rows to load and to store
// (bit b = buffer b), where its segment's step records start, and optionally
// an alias table: 64 bytes, byte b the row whose final value buffer b gets
// (0xFF: its own row).  A step's further destinations whose values nothing
// touches afterwards are stored that way, from the first destination's row,
// instead of by a store record.  The
// records are the steps of the run's phases covering the segment, in phase
// order; steps of one phase touch disjoint positions written by others (the
// phases are hazard-free), so running them one after the other per lane
// gives the phase's result.  Records (32-bit words, first byte the opcode):
//  * kResAdd2 | r0 << 8 | r1 << 16 | d << 24: d = r0 + r1 (fold order r0, r1);
//  * kResCopy | r0 << 8 | r0 << 16 | d << 24: d = r0;
//  * kResChain | m << 8 | s << 16 | d << 24, then ceil(m / 4) words of four
//    row bytes y1..ym: a chain of m 2-source steps each folding the previous
//    result with the next row (acc = s, acc = fold(acc, yi) rounded per step,
//    then d = acc); the intermediate results, which nothing reads later,
//    stay in registers;
//  * kResFold | k << 8 | d << 16, then ceil(k / 4) words of the k >= 2
//    source rows in fold order: d = fold(rows);
//  * kResStore | nd << 8, then nd / 4 words of destination rows (nd a
//    multiple of 4; a list is padded by repeating its last row): each gets
//    the previous record's result (a step with several destinations is its
//    fold, add or copy into the first, then a store into the others).
// Row bytes are packed four per word.
// The records are read 64 words at a time (one word per lane, broadcast with
// v_readlane; the next chunk is loaded while one is run), so no record
// straddles a 64-word chunk; a word 0 ends a chunk early.  The one-word
// records run pipelined: the previous record's result stays in registers (a
// read of the row it wrote takes it from there), so the next record's LDS
// reads go out before the previous result is written to LDS.
constexpr int kResMaxN = 64;  // buffers of a plan the resident kernel takes

struct ResUnit {
    int64_t lo;      // first element of the tile
    uint64_t load;   // rows to load
    uint64_t store;  // rows to store
    int32_t nv;      // 16-byte vectors in the tile, 1..64
    int32_t off;     // first word of the segment's step records
    int32_t nw;      // words of step records (chunk padding included)
    int32_t alias;   // first word of the segment's alias table, or -1
};

constexpr uint32_t kResAdd2 = 0xFE;
constexpr uint32_t kResCopy = 0xFD;
constexpr uint32_t kResChain = 0xFC;
constexpr uint32_t kResFold = 0xFB;
constexpr uint32_t kResStore = 0xFA;

__device__ __forceinline__ int res_byte(uint32_t x, int i) { return int((x >> (8 * i)) & 0xFFu); }

// One 32-bit word of an element vector: the accumulator of a lane that owns
// a word (one fp32 or int32 element, or two bf16 elements) of each row.
template <int DT> struct WAcc;
template <> struct WAcc<DT_F32> {
    float v;
    __device__ __forceinline__ void init(uint32_t x) { v = __uint_as_float(x); }
    __device__ __forceinline__ void add(uint32_t x) { v += __uint_as_float(x); }
    __device__ __forceinline__ uint32_t out() const { return __float_as_uint(v); }
};
template <> struct WAcc<DT_I32> {
    uint32_t v;
    __device__ __forceinline__ void init(uint32_t x) { v = x; }
    __device__ __forceinline__ void add(uint32_t x) { v += x; }
    __device__ __forceinline__ uint32_t out() const { return v; }
};
template <> struct WAcc<DT_BF16> {
    float lo, hi;
    __device__ __forceinline__ void init(uint32_t x) { lo = bf16_lo(x); hi = bf16_hi(x); }
    __device__ __forceinline__ void add(uint32_t x) { lo += bf16_lo(x); hi += bf16_hi(x); }
    __device__ __forceinline__ uint32_t out() const { return bf16_pack(lo, hi); }
};

// What a lane of a W-wave workgroup owns of each row while the records run:
// with one wave its 16-byte vector (row stride 64 vectors), with four waves
// one 32-bit word of its wave's quarter of the row (wave w, lane l: word
// 64 w + l, row stride 256 words).  Every record is element-wise, so the
// waves run the same records on their own words with no barrier between
// records; a quarter row is 256 contiguous bytes, so a wave's LDS accesses
// hit every bank once.
template <int DT, int W> struct ResLane;
template <int DT> struct ResLane<DT, 1> {
    using Word = u32x4;
    using Acc = VAcc<DT>;
    static constexpr int kStride = 64;
};
template <int DT> struct ResLane<DT, 4> {
    using Word = uint32_t;
    using Acc = WAcc<DT>;
    static constexpr int kStride = 256;
};

template <int DT, int W, bool NT>
__global__ __launch_bounds__(64 * W) void resident_kernel(
    const uint64_t* __restrict__ bufs, int32_t n, const ResUnit* __restrict__ units,
    const uint32_t* __restrict__ prog, int64_t nunits) {
    extern __shared__ u32x4 rows[];
    using Word = typename ResLane<DT, W>::Word;
    using Acc = typename ResLane<DT, W>::Acc;
    constexpr int RS = ResLane<DT, W>::kStride;
    constexpr int VEC = Elem<DT>::VEC;
    const int lane = int(threadIdx.x) & 63;
    const int wv = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
    const int64_t unit = int64_t(blockIdx.x);
    if (unit >= nunits) return;  // the same for the whole workgroup
    const ResUnit u = units[unit];
    const bool act = lane < u.nv;
    // lanes past the tile's end read the tile's first vector and store nothing
    const int64_t v = u.lo / VEC + (act ? lane : 0);
    const uint32_t* sp = prog + u.off;
    uint32_t w = lane < u.nw ? sp[lane] : 0u;  // first chunk of step records
    const uint64_t mine = lane < n ? bufs[lane] : 0;
    const uint32_t plo = uint32_t(mine), phi = uint32_t(mine >> 32);
    const uint32_t aw = u.alias >= 0 && lane < 16 ? prog[u.alias + lane] : 0xFFFFFFFFu;
    // the pointers (and the first records) have arrived: the row loads
    // below then go out back to back, with no wait between them
    __builtin_amdgcn_s_waitcnt(0);
    auto at = [&](int b) {
        const uint64_t a =
            (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(phi), b))) << 32) |
            uint32_t(__builtin_amdgcn_readlane(int(plo), b));
        return reinterpret_cast<gvec*>(a) + v;
    };
    // rows b with b % W == wv
    const uint64_t mine_rows = W == 1 ? ~uint64_t(0) : 0x1111111111111111ull << wv;
    for (uint64_t m = u.load & mine_rows; m; m &= m - 1) {
        const int b = __builtin_ctzll(m);
        __builtin_amdgcn_global_load_lds((const AR_GLOBAL void*)(at(b)),
                                         (AR_LDS void*)(rows + b * 64), 16, 0, NT ? 2 : 0);
    }
    if (W == 1) __builtin_amdgcn_s_waitcnt(0);
    else __syncthreads();  // waits for this wave's loads, then for every wave
    // this lane's part of row b is R[b * RS]
    Word* const R = reinterpret_cast<Word*>(rows) + (W == 1 ? lane : wv * 64 + lane);
    {
        Word last{};       // result of the previous one-word record
        int last_row = -1;  // the row it went to (-1: none)
        for (int c0 = 0; c0 < u.nw; c0 += 64) {
            const uint32_t wn = c0 + 64 + lane < u.nw ? sp[c0 + 64 + lane] : 0u;
            const int m = min(64, u.nw - c0);
            int c = 0;
            uint32_t h = uint32_t(__builtin_amdgcn_readlane(int(w), 0));
            Word pa = last, pb = last;  // LDS reads issued for a one-word record
            auto issue = [&]() {
                const uint32_t op = h & 0xFFu;
                if (op == kResAdd2 || op == kResCopy) {
                    pa = R[res_byte(h, 1) * RS];
                    pb = R[res_byte(h, 2) * RS];
                }
            };
            issue();
            while (c < m) {
                const uint32_t op = h & 0xFFu;
                if (op == 0) break;
                if (op == kResAdd2 || op == kResCopy) {
                    const int r0 = res_byte(h, 1), r1 = res_byte(h, 2), d = res_byte(h, 3);
                    const Word a = r0 == last_row ? last : pa;
                    Word out = a;
                    if (op == kResAdd2) {
                        const Word b = r1 == last_row ? last : pb;
                        Acc acc;
                        acc.init(a);
                        acc.add(b);
                        out = acc.out();
                    }
                    c += 1;
                    h = c < m ? uint32_t(__builtin_amdgcn_readlane(int(w), c)) : 0u;
                    issue();  // the next record's reads, before this write
                    R[d * RS] = out;
                    last = out;
                    last_row = d;
                } else if (op == kResChain) {
                    const int mm = res_byte(h, 1), d = res_byte(h, 3);
                    Word cur = R[res_byte(h, 2) * RS];
                    for (int i0 = 0; i0 < mm; i0 += 8) {
                        const uint32_t wa = uint32_t(__builtin_amdgcn_readlane(int(w), c + 1 + (i0 >> 2)));
                        const uint32_t wb =
                            i0 + 4 < mm ? uint32_t(__builtin_amdgcn_readlane(int(w), c + 2 + (i0 >> 2))) : 0u;
                        Word y[8];
#pragma unroll
                        for (int j = 0; j < 8; ++j)
                            if (i0 + j < mm) y[j] = R[res_byte(j < 4 ? wa : wb, j & 3) * RS];
#pragma unroll
                        for (int j = 0; j < 8; ++j)
                            if (i0 + j < mm) {
                                Acc acc;
                                acc.init(cur);
                                acc.add(y[j]);
                                cur = acc.out();
                            }
                    }
                    c += 1 + (mm + 3) / 4;
                    h = c < m ? uint32_t(__builtin_amdgcn_readlane(int(w), c)) : 0u;
                    issue();  // the next record's reads, before this write
                    R[d * RS] = cur;
                    last = cur;
                    last_row = d;
                } else if (op == kResFold) {
                    const int k = res_byte(h, 1), d = res_byte(h, 2);
                    Acc acc;
                    const int kg = k >> 2;  // full groups of four sources
                    for (int g = 0; g < kg; ++g) {
                        const uint32_t x = uint32_t(__builtin_amdgcn_readlane(int(w), c + 1 + g));
                        const Word a0 = R[res_byte(x, 0) * RS];
                        const Word a1 = R[res_byte(x, 1) * RS];
                        const Word a2 = R[res_byte(x, 2) * RS];
                        const Word a3 = R[res_byte(x, 3) * RS];
                        if (g == 0) acc.init(a0);
                        else acc.add(a0);
                        acc.add(a1);
                        acc.add(a2);
                        acc.add(a3);
                    }
                    const int rem = k & 3;
                    if (rem) {
                        const uint32_t x = uint32_t(__builtin_amdgcn_readlane(int(w), c + 1 + kg));
                        const Word a0 = R[res_byte(x, 0) * RS];
                        const Word a1 = R[res_byte(x, rem > 1 ? 1 : 0) * RS];
                        const Word a2 = R[res_byte(x, rem > 2 ? 2 : 0) * RS];
                        if (kg == 0) acc.init(a0);
                        else acc.add(a0);
                        if (rem > 1) acc.add(a1);
                        if (rem > 2) acc.add(a2);
                    }
                    const Word out = acc.out();
                    c += 1 + ((k + 3) >> 2);
                    h = c < m ? uint32_t(__builtin_amdgcn_readlane(int(w), c)) : 0u;
                    issue();  // the next record's reads, before this write
                    R[d * RS] = out;
                    last = out;
                    last_row = d;
                } else {  // kResStore: the previous result into nd rows
                    const int nq = res_byte(h, 1) >> 2;
                    for (int j = 0; j < nq; ++j) {
                        const uint32_t x = uint32_t(__builtin_amdgcn_readlane(int(w), c + 1 + j));
                        R[res_byte(x, 0) * RS] = last;
                        R[res_byte(x, 1) * RS] = last;
                        R[res_byte(x, 2) * RS] = last;
                        R[res_byte(x, 3) * RS] = last;
                    }
                    c += 1 + nq;
                    h = c < m ? uint32_t(__builtin_amdgcn_readlane(int(w), c)) : 0u;
                    issue();
                }
            }
            w = wn;
        }
    }
    if (W > 1) __syncthreads();  // the rows are final
    uint64_t m = u.store & mine_rows;
    while (m) {
        int b[8];
        u32x4 x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            b[j] = m ? __builtin_ctzll(m) : -1;
            m &= m - 1;
            if (b[j] >= 0) {
                const int r = res_byte(uint32_t(__builtin_amdgcn_readlane(int(aw), b[j] >> 2)), b[j] & 3);
                x[j] = rows[(r == 0xFF ? b[j] : r) * 64 + lane];
            }
        }
        if (act) {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (b[j] >= 0) vstore<NT>(at(b[j]), x[j]);
        }
    }
}

// ------------------------------------------------------------------------
// Streamed resident kernel: the resident form for plans with more buffers
// than rows fit in LDS.  A workgroup still owns one 1 KiB tile of a segment,
// but its LDS holds S slots of 1 KiB instead of a row per buffer: the host
// turns the segment's steps into values (a copy names its source's value, a
// step with k >= 2 sources a new one), computes each value once its inputs
// are there, in an order that finishes one subtree of folds before the next
// (depth first), gives every value a slot from its load or fold to its last
// use, and stores each buffer's final value as soon as it is computed.  The
// buffer rows a segment reads before writing are loaded into slots up to
// kStreamAhead rows ahead of their first use.  Every fold runs on the same
// values in the same source order as in the plan, so the results are the
// same bits.
//
// Its W waves (1 or 4) run independently, with no barrier after the
// workgroup has copied the n buffer pointers and the unit's records into LDS
// behind the slots: one wave owns the whole tile (16 bytes a lane), four
// waves a 256-byte quarter each (wave w, lane l: bytes 256 w + 4 l); each
// loads its part of every row straight into LDS (global_load_lds), runs every
// record on it and stores it.  A load or store record's lanes look up its
// entries' pointers in LDS at once.
// Besides add (kResAdd2) and fold (kResFold) records over slot bytes:
//  * kResLoad | c << 8, then c words slot | buffer << 8: load the buffers'
//    quarter rows into the slots (in flight until a wait);
//  * kResWait | m << 8: wait until at most m of the wave's row loads and
//    stores are outstanding (the kernel may wait for more).  Loads finish in
//    the order they were issued, stores in any order relative to them, so
//    a load followed by m loads is done once at most m operations remain;
//  * kResPut | c << 8 | slot << 16, then (c + 1) / 2 words of two 16-bit
//    buffer numbers: store the slot's value into the buffers.
constexpr uint32_t kResLoad = 0xF9;
constexpr uint32_t kResWait = 0xF8;
constexpr uint32_t kResPut = 0xF7;
constexpr int kStreamMaxSlots = 64;
constexpr int kStreamMaxN = 4096;  // buffers: their pointers take 8 n bytes of LDS

// s_waitcnt vmcnt(V) with the other counters not waited for (gfx9 encoding:
// vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8)
template <int V>
__device__ __forceinline__ void wait_vm() {
    __builtin_amdgcn_s_waitcnt((V & 15) | ((V >> 4) << 14) | (7 << 4) | (15 << 8));
}

// wait until at most m vector memory operations are outstanding (m rounded
// down to a multiple of four below 64, or to 0, 1 or 2)
__device__ __forceinline__ void wait_vm_at_most(int m) {
    switch (m >= 60 ? 15 : m >> 2) {
        case 15: wait_vm<60>(); break;
        case 14: wait_vm<56>(); break;
        case 13: wait_vm<52>(); break;
        case 12: wait_vm<48>(); break;
        case 11: wait_vm<44>(); break;
        case 10: wait_vm<40>(); break;
        case 9: wait_vm<36>(); break;
        case 8: wait_vm<32>(); break;
        case 7: wait_vm<28>(); break;
        case 6: wait_vm<24>(); break;
        case 5: wait_vm<20>(); break;
        case 4: wait_vm<16>(); break;
        case 3: wait_vm<12>(); break;
        case 2: wait_vm<8>(); break;
        case 1: wait_vm<4>(); break;
        default:
            if (m >= 2) wait_vm<2>();
            else if (m == 1) wait_vm<1>();
            else wait_vm<0>();
    }
}

template <int DT, int W, bool NT>
__global__ __launch_bounds__(64 * W) void stream_kernel(
    const uint64_t* __restrict__ bufs, int32_t n, int32_t slots,
    const ResUnit* __restrict__ units, const uint32_t* __restrict__ prog, int64_t nunits) {
    extern __shared__ u32x4 rows[];
    using Word = typename ResLane<DT, W>::Word;
    using Acc = typename ResLane<DT, W>::Acc;
    constexpr int RS = ResLane<DT, W>::kStride;  // words per slot
    constexpr int BYTES = W == 1 ? 16 : 4;       // bytes a lane owns of the tile
    const int lane = int(threadIdx.x) & 63;
    const int wv = __builtin_amdgcn_readfirstlane(int(threadIdx.x) >> 6);
    const int64_t unit = int64_t(blockIdx.x);
    if (unit >= nunits) return;  // the same for the whole workgroup
    const ResUnit u = units[unit];
    // behind the slots: the buffer pointers (a record's lanes look up the
    // pointers of its entries at once) and the unit's records, copied once
    // before any row load: reading the records from memory as they run
    // would make every 64-word chunk wait for all row loads in flight
    uint64_t* const ptab = reinterpret_cast<uint64_t*>(rows + slots * 64);
    uint32_t* const lprog = reinterpret_cast<uint32_t*>(ptab + n);
    for (int i = int(threadIdx.x); i < n; i += 64 * W) ptab[i] = bufs[i];
    for (int i = int(threadIdx.x); i < u.nw; i += 64 * W) lprog[i] = prog[u.off + i];
    __syncthreads();
    // this lane's part of the tile; lanes past the tile's end read its first
    // bytes and store nothing
    const int wb = wv * 256 + lane * BYTES;
    const bool act = wb < u.nv * 16;
    const int64_t goff = u.lo * int64_t(Elem<DT>::VEC == 8 ? 2 : 4) + (act ? wb : 0);
    Word* const R = reinterpret_cast<Word*>(rows) + (W == 1 ? lane : wv * 64 + lane);  // slot s: R[s * RS]
    uint32_t w = lane < u.nw ? lprog[lane] : 0u;  // first chunk of records
    auto gptr = [&](uint64_t base) {  // this lane's part of a buffer's tile
        return (AR_GLOBAL Word*)(base + uint64_t(goff));
    };
    // the pointer of entry j of the record at word c (entry j in lane
    // c + 1 + j), held by lane c + 1 + j
    auto entry_ptr = [&](const uint64_t p, int j, int c) {
        return (uint64_t(uint32_t(__builtin_amdgcn_readlane(int(uint32_t(p >> 32)), c + 1 + j))) << 32) |
               uint32_t(__builtin_amdgcn_readlane(int(uint32_t(p)), c + 1 + j));
    };
    for (int c0 = 0; c0 < u.nw; c0 += 64) {
        const uint32_t wn = c0 + 64 + lane < u.nw ? lprog[c0 + 64 + lane] : 0u;
        const int m = min(64, u.nw - c0);
        int c = 0;
        while (c < m) {
            const uint32_t h = uint32_t(__builtin_amdgcn_readlane(int(w), c));
            const uint32_t op = h & 0xFFu;
            if (op == 0) break;
            if (op == kResAdd2) {
                Acc acc;
                acc.init(R[res_byte(h, 1) * RS]);
                acc.add(R[res_byte(h, 2) * RS]);
                R[res_byte(h, 3) * RS] = acc.out();
                c += 1;
            } else if (op == kResFold) {
                const int k = res_byte(h, 1), d = res_byte(h, 2);
                Acc acc;
                const int kg = k >> 2;  // full groups of four sources
                for (int g = 0; g < kg; ++g) {
                    const uint32_t x = uint32_t(__builtin_amdgcn_readlane(int(w), c + 1 + g));
                    const Word a0 = R[res_byte(x, 0) * RS];
                    const Word a1 = R[res_byte(x, 1) * RS];
                    const Word a2 = R[res_byte(x, 2) * RS];
                    const Word a3 = R[res_byte(x, 3) * RS];
                    if (g == 0) acc.init(a0);
                    else acc.add(a0);
                    acc.add(a1);
                    acc.add(a2);
                    acc.add(a3);
                }
                const int rem = k & 3;
                if (rem) {
                    const uint32_t x = uint32_t(__builtin_amdgcn_readlane(int(w), c + 1 + kg));
                    const Word a0 = R[res_byte(x, 0) * RS];
                    const Word a1 = R[res_byte(x, rem > 1 ? 1 : 0) * RS];
                    const Word a2 = R[res_byte(x, rem > 2 ? 2 : 0) * RS];
                    if (kg == 0) acc.init(a0);
                    else acc.add(a0);
                    if (rem > 1) acc.add(a1);
                    if (rem > 2) acc.add(a2);
                }
                R[d * RS] = acc.out();
                c += 1 + ((k + 3) >> 2);
            } else if (op == kResLoad) {
                const int cnt = res_byte(h, 1);
                const bool mine = lane > c && lane <= c + cnt;  // this lane's word is an entry
                const uint64_t p = ptab[mine ? w >> 8 : 0u];
                for (int j = 0; j < cnt; ++j) {
                    const uint32_t x = uint32_t(__builtin_amdgcn_readlane(int(w), c + 1 + j));
                    const AR_GLOBAL void* src = (const AR_GLOBAL void*)(gptr(entry_ptr(p, j, c)));
                    AR_LDS void* dst =
                        (AR_LDS void*)((AR_LDS char*)(rows) + (x & 0xFFu) * 1024u + uint32_t(wv) * 256u);
                    if constexpr (W == 1) __builtin_amdgcn_global_load_lds(src, dst, 16, 0, NT ? 2 : 0);
                    else __builtin_amdgcn_global_load_lds(src, dst, 4, 0, NT ? 2 : 0);
                }
                c += 1 + cnt;
            } else if (op == kResWait) {
                wait_vm_at_most(res_byte(h, 1));
                c += 1;
            } else {  // kResPut
                const int cnt = res_byte(h, 1);
                const Word val = R[res_byte(h, 2) * RS];
                const bool mine = lane > c && lane <= c + ((cnt + 1) >> 1);
                const uint64_t p0 = ptab[mine ? w & 0xFFFFu : 0u];
                const uint64_t p1 = ptab[mine ? w >> 16 : 0u];
                for (int j = 0; j < cnt; ++j) {
                    const uint64_t base = entry_ptr(j & 1 ? p1 : p0, j >> 1, c);
                    if (act) {
                        if constexpr (NT) __builtin_nontemporal_store(val, gptr(base));
                        else *gptr(base) = val;
                    }
                }
                c += 1 + ((cnt + 1) >> 1);
            }
        }
        w = wn;
    }
}

}  // namespace arp
