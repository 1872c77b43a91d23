// C ABI: plan creation, destruction, introspection and error reporting.
// Everything here is host code and makes no HIP call.
#include <algorithm>
#include <climits>
#include <new>
#include <stdexcept>
#include <string>

#include "internal.hpp"

namespace arp {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }
void clear_error() { g_last_error.clear(); }
ar_status fail(ar_status s, const std::string& msg) {
    g_last_error = msg;
    return s;
}

static int32_t esize_of(int32_t dtype) {
    switch (dtype) {
        case AR_F32: return 4;
        case AR_I32: return 4;
        case AR_BF16: return 2;
        default: return 0;
    }
}

// Upper bound on expanded steps; beyond it creation is refused.
static constexpr int64_t kMaxSteps = int64_t(1) << 26;

static int64_t estimate_steps(int32_t kind, int64_t n,
                              const std::vector<int32_t>& fan) {
    switch (kind) {
        case AR_RING: return 2 * (n - 1) * n;
        case AR_RHD: { int64_t k = 0; while ((int64_t(1) << k) < n) ++k; return 2 * k * n + 2 * n; }
        case AR_CPS: return n * n;
        case AR_RB: return n;
        case AR_TREE: {
            int64_t s = 0;
            for (int32_t f : fan) s += n * f;
            return s;
        }
        default: return 0;
    }
}

template <class F>
static ar_status guarded(F&& f) {
    try {
        return f();
    } catch (const std::bad_alloc&) {
        return fail(AR_ERR_OOM, "host allocation failed");
    } catch (const Unsupported& e) {
        return fail(AR_ERR_UNSUPPORTED, e.what());
    } catch (const std::invalid_argument& e) {
        return fail(AR_ERR_INVALID_ARG, e.what());
    } catch (const std::exception& e) {
        return fail(AR_ERR_INTERNAL, e.what());
    } catch (...) {
        return fail(AR_ERR_INTERNAL, "unknown exception");
    }
}

}  // namespace arp

using namespace arp;

AR_EXPORT ar_status ar_plan_create(int32_t n, int64_t N, int32_t dtype,
                                   const ar_topology* topo, ar_plan** out) {
    clear_error();
    if (!out) return fail(AR_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (!topo) return fail(AR_ERR_INVALID_ARG, "topo is NULL");
    if (n < 1 || n > 65536)
        return fail(AR_ERR_INVALID_ARG, "n must be in [1, 65536]");
    if (N < 0) return fail(AR_ERR_INVALID_ARG, "N must be >= 0");
    const int32_t es = esize_of(dtype);
    if (!es) return fail(AR_ERR_INVALID_ARG, "unknown dtype");
    if (N > INT64_MAX / es)
        return fail(AR_ERR_INVALID_ARG, "N * element size overflows");
    std::vector<int32_t> fan;
    switch (topo->kind) {
        case AR_RING: case AR_RHD: case AR_CPS: case AR_RB: break;
        case AR_TREE: {
            if (topo->num_levels < 1 || !topo->fanin)
                return fail(AR_ERR_INVALID_ARG, "tree needs num_levels >= 1 fan-ins");
            if (topo->num_levels > 64)
                return fail(AR_ERR_INVALID_ARG, "too many tree levels");
            int64_t prod = 1;
            for (int32_t l = 0; l < topo->num_levels; ++l) {
                const int32_t f = topo->fanin[l];
                if (f < 1) return fail(AR_ERR_INVALID_ARG, "fan-in must be >= 1");
                prod *= f;
                if (prod > n) break;
                fan.push_back(f);
            }
            if (prod != n)
                return fail(AR_ERR_INVALID_ARG, "product of fan-ins must equal n");
            break;
        }
        default:
            return fail(AR_ERR_INVALID_ARG, "unknown plan kind");
    }
    if (estimate_steps(topo->kind, n, fan) > kMaxSteps)
        return fail(AR_ERR_UNSUPPORTED, "plan would exceed 2^26 steps");
    return guarded([&]() -> ar_status {
        ar_plan* p = new ar_plan();
        p->n = n;
        p->N = N;
        p->dtype = dtype;
        p->esize = es;
        p->kind = topo->kind;
        p->fanin = fan;
        try {
            switch (topo->kind) {
                case AR_RING: expand_ring(*p); break;
                case AR_RHD: expand_rhd(*p); break;
                case AR_CPS: expand_cps(*p); break;
                case AR_TREE: expand_tree(*p); break;
                case AR_RB: expand_rb(*p); break;
            }
            validate_phases(*p);
        } catch (...) {
            delete p;
            throw;
        }
        *out = p;
        return AR_OK;
    });
}

AR_EXPORT ar_status ar_plan_create_gentree(int64_t N, int32_t dtype, int32_t num_nodes,
                                           const int32_t* nchild, ar_plan** out) {
    clear_error();
    if (!out) return fail(AR_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (num_nodes < 1 || !nchild)
        return fail(AR_ERR_INVALID_ARG, "need num_nodes >= 1 child counts");
    if (N < 0) return fail(AR_ERR_INVALID_ARG, "N must be >= 0");
    const int32_t es = esize_of(dtype);
    if (!es) return fail(AR_ERR_INVALID_ARG, "unknown dtype");
    if (N > INT64_MAX / es)
        return fail(AR_ERR_INVALID_ARG, "N * element size overflows");
    std::vector<int32_t> counts(nchild, nchild + num_nodes);
    const int64_t n = gentree_servers(counts);
    if (n < 1)
        return fail(AR_ERR_INVALID_ARG, "child counts do not describe exactly one tree");
    if (n > 65536) return fail(AR_ERR_INVALID_ARG, "more than 65536 servers");
    // size guard: every switch lists, per block, one holder per child
    {
        int64_t work = 0;
        for (int32_t c : counts) work += int64_t(c) * n;
        if (work > (int64_t(1) << 28))
            return fail(AR_ERR_UNSUPPORTED, "tree too large (children x servers > 2^28)");
    }
    return guarded([&]() -> ar_status {
        ar_plan* p = new ar_plan();
        try {
            p->n = int32_t(n);
            p->N = N;
            p->dtype = dtype;
            p->esize = es;
            p->kind = AR_GENTREE;
            expand_gentree(*p, counts);
            validate_phases(*p);
        } catch (...) {
            delete p;
            throw;
        }
        *out = p;
        return AR_OK;
    });
}

AR_EXPORT ar_status ar_plan_create_custom(int32_t n, int64_t N, int32_t dtype,
                                          const ar_step* steps, int64_t nsteps,
                                          ar_plan** out) {
    clear_error();
    if (!out) return fail(AR_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (n < 1 || n > 65536)
        return fail(AR_ERR_INVALID_ARG, "n must be in [1, 65536]");
    if (N < 0) return fail(AR_ERR_INVALID_ARG, "N must be >= 0");
    const int32_t es = esize_of(dtype);
    if (!es) return fail(AR_ERR_INVALID_ARG, "unknown dtype");
    if (N > INT64_MAX / es)
        return fail(AR_ERR_INVALID_ARG, "N * element size overflows");
    if (nsteps < 0 || nsteps > kMaxSteps)
        return fail(AR_ERR_INVALID_ARG, "nsteps must be in [0, 2^26]");
    if (nsteps > 0 && !steps) return fail(AR_ERR_INVALID_ARG, "steps is NULL");
    int32_t max_phase = -1;
    for (int64_t i = 0; i < nsteps; ++i) {
        const ar_step& s = steps[i];
        const std::string at = "step " + std::to_string(i) + ": ";
        if (s.phase < 0) return fail(AR_ERR_INVALID_ARG, at + "phase < 0");
        if (s.op != AR_OP_REDUCE && s.op != AR_OP_COPY)
            return fail(AR_ERR_INVALID_ARG, at + "unknown op");
        if (s.dst < 0 || s.dst >= n)
            return fail(AR_ERR_INVALID_ARG, at + "dst out of range");
        if (s.nsrc < 1 || s.nsrc > n * 64)
            return fail(AR_ERR_INVALID_ARG, at + "bad source count");
        if (s.op == AR_OP_COPY && s.nsrc != 1)
            return fail(AR_ERR_INVALID_ARG, at + "a copy has exactly one source");
        if (!s.srcs) return fail(AR_ERR_INVALID_ARG, at + "srcs is NULL");
        for (int32_t t = 0; t < s.nsrc; ++t)
            if (s.srcs[t] < 0 || s.srcs[t] >= n)
                return fail(AR_ERR_INVALID_ARG, at + "source out of range");
        if (s.begin < 0 || s.begin > s.end || s.end > N)
            return fail(AR_ERR_INVALID_ARG, at + "range outside [0, N]");
        max_phase = std::max(max_phase, s.phase);
    }
    return guarded([&]() -> ar_status {
        std::vector<int64_t> order(static_cast<size_t>(nsteps));
        for (int64_t i = 0; i < nsteps; ++i) order[size_t(i)] = i;
        std::stable_sort(order.begin(), order.end(), [&](int64_t a, int64_t b) {
            return steps[a].phase < steps[b].phase;
        });
        std::vector<char> seen(size_t(max_phase + 1), 0);
        for (int64_t i = 0; i < nsteps; ++i) seen[size_t(steps[i].phase)] = 1;
        for (int32_t ph = 0; ph <= max_phase; ++ph)
            if (!seen[size_t(ph)])
                return fail(AR_ERR_INVALID_ARG,
                            "phase " + std::to_string(ph) + " has no step");
        ar_plan* p = new ar_plan();
        try {
            p->n = n;
            p->N = N;
            p->dtype = dtype;
            p->esize = es;
            p->kind = -1;
            for (int64_t i : order) {
                const ar_step& s = steps[i];
                p->add(s.phase, s.op, s.dst,
                       std::vector<int32_t>(s.srcs, s.srcs + s.nsrc), s.begin,
                       s.end);
            }
            p->finish_phases();
            validate_phases(*p);
        } catch (...) {
            delete p;
            throw;
        }
        *out = p;
        return AR_OK;
    });
}

AR_EXPORT ar_status ar_plan_destroy(ar_plan* plan) {
    clear_error();
    if (!plan) return AR_OK;
    exec_release(*plan);
    delete plan;
    return AR_OK;
}

AR_EXPORT ar_status ar_plan_info(const ar_plan* plan, int32_t* n, int64_t* N,
                                 int32_t* dtype, int32_t* num_phases,
                                 int64_t* num_steps) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    if (n) *n = plan->n;
    if (N) *N = plan->N;
    if (dtype) *dtype = plan->dtype;
    if (num_phases) *num_phases = plan->num_phases();
    if (num_steps) *num_steps = int64_t(plan->steps.size());
    return AR_OK;
}

AR_EXPORT ar_status ar_plan_get_step(const ar_plan* plan, int64_t i,
                                     ar_step* out) {
    clear_error();
    if (!plan || !out) return fail(AR_ERR_INVALID_ARG, "NULL argument");
    if (i < 0 || i >= int64_t(plan->steps.size()))
        return fail(AR_ERR_INVALID_ARG, "step index out of range");
    const Step& s = plan->steps[size_t(i)];
    out->phase = s.phase;
    out->op = s.op;
    out->dst = s.dst;
    out->nsrc = s.nsrc;
    out->srcs = plan->srcs.data() + s.src_off;
    out->begin = s.begin;
    out->end = s.end;
    return AR_OK;
}

AR_EXPORT ar_status ar_plan_phase_info(const ar_plan* plan, int32_t phase,
                                       int32_t* op, int64_t* first_step,
                                       int64_t* num_steps, int64_t* bytes) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    if (phase < 0 || phase >= plan->num_phases())
        return fail(AR_ERR_INVALID_ARG, "phase out of range");
    const int64_t s0 = plan->phase_first[size_t(phase)];
    const int64_t s1 = plan->phase_first[size_t(phase) + 1];
    int32_t o = AR_OP_COPY;
    int64_t b = 0;
    for (int64_t i = s0; i < s1; ++i) {
        const Step& s = plan->steps[size_t(i)];
        if (s.op == OP_REDUCE) o = AR_OP_REDUCE;
        b += step_bytes(*plan, s);
    }
    if (op) *op = o;
    if (first_step) *first_step = s0;
    if (num_steps) *num_steps = s1 - s0;
    if (bytes) *bytes = b;
    return AR_OK;
}

AR_EXPORT ar_status ar_plan_owner(const ar_plan* plan, int32_t p,
                                  int64_t* begin, int64_t* end) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    if (p < 0 || p >= plan->n) return fail(AR_ERR_INVALID_ARG, "p out of range");
    if (plan->owner_begin.empty())
        return fail(AR_ERR_UNSUPPORTED, "custom plans have no owner map");
    if (plan->owner_begin[size_t(p)] < 0)
        return fail(AR_ERR_UNSUPPORTED, "this processor's blocks are not contiguous");
    if (begin) *begin = plan->owner_begin[size_t(p)];
    if (end) *end = plan->owner_end[size_t(p)];
    return AR_OK;
}

AR_EXPORT ar_status ar_plan_bytes(const ar_plan* plan, int64_t* reduce_bytes,
                                  int64_t* copy_bytes) {
    clear_error();
    if (!plan) return fail(AR_ERR_INVALID_ARG, "plan is NULL");
    int64_t r = 0, c = 0;
    for (const Step& s : plan->steps)
        (s.op == OP_REDUCE ? r : c) += step_bytes(*plan, s);
    if (reduce_bytes) *reduce_bytes = r;
    if (copy_bytes) *copy_bytes = c;
    return AR_OK;
}

AR_EXPORT const char* ar_status_string(ar_status s) {
    switch (s) {
        case AR_OK: return "AR_OK";
        case AR_ERR_INVALID_ARG: return "AR_ERR_INVALID_ARG";
        case AR_ERR_UNSUPPORTED: return "AR_ERR_UNSUPPORTED";
        case AR_ERR_OOM: return "AR_ERR_OOM";
        case AR_ERR_HIP: return "AR_ERR_HIP";
        case AR_ERR_INTERNAL: return "AR_ERR_INTERNAL";
        default: return "AR_ERR_UNKNOWN";
    }
}

AR_EXPORT const char* ar_last_error(void) { return g_last_error.c_str(); }
