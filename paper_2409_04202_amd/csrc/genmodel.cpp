// GenModel on one GPU: the terms of a plan's predicted time, with one cache
// or a list of cache tiers, and the plan kind of smallest predicted time
// among the candidates (the model's use in plan selection, Section 3.4 and
// Algorithm 2, with the terms a single GPU has).  Host only; no HIP call.
#include <algorithm>
#include <array>
#include <cstring>
#include <new>
#include <set>
#include <stdexcept>
#include <string>
#include <tuple>
#include <vector>

#include "internal.hpp"

namespace arp {

namespace {

using Range = std::tuple<int32_t, int64_t, int64_t>;  // (buffer, begin, end)

// terms[0..AR_GENMODEL_TERMS) of plan p; see ar_genmodel_terms.
void plan_terms(const Plan& p, int64_t cache_bytes, double* t) {
    const double footprint = double(p.n) * double(p.N) * double(p.esize);
    const bool fits = footprint <= double(cache_bytes);
    double K = 0, Dh = 0, Dc = 0, Bh = 0, Bc = 0;
    std::set<Range> prev_written;
    int64_t prev_bytes = 0;
    const int32_t P = p.num_phases();
    for (int32_t ph = 0; ph < P; ++ph) {
        const int64_t s0 = p.phase_first[size_t(ph)], s1 = p.phase_first[size_t(ph) + 1];
        if (s1 <= s0) continue;
        int32_t widest = 0;
        bool reduce = false;
        std::set<Range> seen, written;
        int64_t wbytes = 0;
        double h = 0, c = 0;
        for (int64_t i = s0; i < s1; ++i) {
            const Step& st = p.steps[size_t(i)];
            widest = std::max(widest, st.nsrc);
            reduce = reduce || st.op == OP_REDUCE;
            const int64_t len = (st.end - st.begin) * p.esize;
            for (int32_t j = 0; j < st.nsrc; ++j) {
                const Range key{p.srcs[size_t(st.src_off + j)], st.begin, st.end};
                // the first read of a range in the phase comes from HBM unless
                // the whole footprint fits the cache or the previous phase
                // wrote it (and no more than the cache holds); repeats hit
                const bool cached = fits || seen.count(key) ||
                                    (prev_bytes <= cache_bytes && prev_written.count(key));
                (cached ? c : h) += double(len);
                seen.insert(key);
            }
            (fits ? c : h) += double(len);  // the write
            written.insert(Range{st.dst, st.begin, st.end});
            wbytes += len;
        }
        K += widest;
        if (reduce) {
            Dh += h;
            Dc += c;
        } else {
            Bh += h;
            Bc += c;
        }
        prev_written.swap(written);
        prev_bytes = wbytes;
    }
    t[0] = double(P);
    t[1] = K;
    t[2] = Dh;
    t[3] = Dc;
    t[4] = Bh;
    t[5] = Bc;
}

// terms[0..4 + 2 * tiers) of plan p with the cache tiers cache_bytes[0..tiers)
// (strictly decreasing): A, K, then the reduce bytes served from HBM and
// from each tier, then the copy bytes the same way (see
// ar_genmodel_terms_tiered).  An access is served from the smallest tier
// under whose size the one-cache rule classes it as cached: that rule is
// monotone in the size, so tier i's bytes are what size i classes as cached
// less what size i + 1 does.
void tiered_terms(const Plan& p, int32_t tiers, const int64_t* cache_bytes, double* t) {
    std::vector<std::array<double, AR_GENMODEL_TERMS>> per(size_t(tiers) + 1);
    for (int32_t i = 0; i < tiers; ++i) plan_terms(p, cache_bytes[i], per[size_t(i)].data());
    per[size_t(tiers)].fill(0.0);  // a size-0 "tier" below the last: nothing cached
    t[0] = per[0][0];
    t[1] = per[0][1];
    t[2] = per[0][2];                          // reduce bytes from HBM
    t[3 + tiers] = per[0][4];                  // copy bytes from HBM
    for (int32_t i = 0; i < tiers; ++i) {
        t[3 + i] = per[size_t(i)][3] - per[size_t(i) + 1][3];
        t[4 + tiers + i] = per[size_t(i)][5] - per[size_t(i) + 1][5];
    }
}

// Ordered factorisations of n into 2..max_levels factors >= 2, each list
// built from the smallest first factor up (depth first).
void factorizations(int32_t rest, int32_t max_levels, std::vector<int32_t>& cur,
                    std::vector<std::vector<int32_t>>& out) {
    if (rest == 1) {
        if (cur.size() >= 2) out.push_back(cur);
        return;
    }
    if (int32_t(cur.size()) == max_levels) return;
    for (int32_t f = 2; f <= rest; ++f)
        if (rest % f == 0) {
            cur.push_back(f);
            factorizations(rest / f, max_levels, cur, out);
            cur.pop_back();
        }
}

}  // namespace

}  // namespace arp

using namespace arp;

AR_EXPORT ar_status ar_genmodel_terms(const ar_plan* plan, int64_t cache_bytes, double* terms) {
    clear_error();
    if (!plan || !terms) return fail(AR_ERR_INVALID_ARG, "NULL argument");
    if (cache_bytes < 0) return fail(AR_ERR_INVALID_ARG, "cache_bytes < 0");
    try {
        plan_terms(*plan, cache_bytes, terms);
        return AR_OK;
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}

// Whether cache_bytes[0..tiers) is a valid tier list: 1..AR_GENMODEL_MAX_TIERS
// sizes, each >= 0, strictly decreasing.
static bool valid_tiers(int32_t tiers, const int64_t* cache_bytes) {
    if (tiers < 1 || tiers > AR_GENMODEL_MAX_TIERS || !cache_bytes) return false;
    for (int32_t i = 0; i < tiers; ++i)
        if (cache_bytes[i] < 0 || (i > 0 && cache_bytes[i] >= cache_bytes[i - 1])) return false;
    return true;
}

AR_EXPORT ar_status ar_genmodel_terms_tiered(const ar_plan* plan, int32_t tiers,
                                             const int64_t* cache_bytes, double* terms) {
    clear_error();
    if (!plan || !terms) return fail(AR_ERR_INVALID_ARG, "NULL argument");
    if (!valid_tiers(tiers, cache_bytes))
        return fail(AR_ERR_INVALID_ARG, "bad tier count or sizes (decreasing, >= 0)");
    try {
        tiered_terms(*plan, tiers, cache_bytes, terms);
        return AR_OK;
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}

AR_EXPORT ar_status ar_genmodel_select(int32_t n, int64_t N, int32_t dtype, const double* params,
                                       int64_t cache_bytes, int32_t max_levels, int32_t* kind,
                                       int32_t* num_levels, int32_t* fanin, double* seconds) {
    clear_error();
    if (cache_bytes < 0) return fail(AR_ERR_INVALID_ARG, "bad n, N, cache_bytes or max_levels");
    return ar_genmodel_select_tiered(n, N, dtype, params, 1, &cache_bytes, max_levels, kind,
                                     num_levels, fanin, seconds);
}

AR_EXPORT ar_status ar_genmodel_select_tiered(int32_t n, int64_t N, int32_t dtype,
                                              const double* params, int32_t tiers,
                                              const int64_t* cache_bytes, int32_t max_levels,
                                              int32_t* kind, int32_t* num_levels,
                                              int32_t* fanin, double* seconds) {
    clear_error();
    if (!params || !kind || !num_levels || !fanin || !seconds)
        return fail(AR_ERR_INVALID_ARG, "NULL argument");
    if (n < 1 || N < 0 || !valid_tiers(tiers, cache_bytes) || max_levels < 2 || max_levels > 32)
        return fail(AR_ERR_INVALID_ARG, "bad n, N, cache_bytes or max_levels");
    const int32_t nterms = 4 + 2 * tiers;
    try {
        struct Cand {
            int32_t kind;
            std::vector<int32_t> fan;
        };
        std::vector<Cand> cands{{AR_RING, {}}, {AR_CPS, {}}, {AR_RHD, {}}};
        std::vector<std::vector<int32_t>> facs;
        std::vector<int32_t> cur;
        factorizations(n, max_levels, cur, facs);
        for (auto& f : facs) cands.push_back({AR_TREE, f});
        bool found = false;
        double best = 0;
        size_t best_i = 0;
        for (size_t i = 0; i < cands.size(); ++i) {
            const ar_topology topo{cands[i].kind, int32_t(cands[i].fan.size()),
                                   cands[i].fan.empty() ? nullptr : cands[i].fan.data()};
            ar_plan* p = nullptr;
            const ar_status s = ar_plan_create(n, N, dtype, &topo, &p);
            if (s == AR_ERR_UNSUPPORTED || s == AR_ERR_OOM) continue;  // too large a plan
            if (s != AR_OK) return s;  // bad arguments: ar_last_error says which
            double t[4 + 2 * AR_GENMODEL_MAX_TIERS];
            try {
                tiered_terms(*p, tiers, cache_bytes, t);
            } catch (...) {
                ar_plan_destroy(p);
                throw;
            }
            ar_plan_destroy(p);
            double pred = 0;
            for (int j = 0; j < nterms; ++j) pred += params[j] * t[j];
            if (!found || pred < best) {
                found = true;
                best = pred;
                best_i = i;
            }
        }
        clear_error();
        if (!found) return fail(AR_ERR_UNSUPPORTED, "no candidate plan could be built");
        *kind = cands[best_i].kind;
        *num_levels = int32_t(cands[best_i].fan.size());
        std::copy(cands[best_i].fan.begin(), cands[best_i].fan.end(), fanin);
        *seconds = best;
        return AR_OK;
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    }
}
