// Host-side plan representation and expanders (no HIP).
//
// A plan is a list of steps sorted by phase.  Steps of one phase are
// independent (checked by validate_phases), so a phase can be executed as
// one batched launch.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace arp {

enum Op : int32_t { OP_REDUCE = 0, OP_COPY = 1 };

struct Step {
    int32_t phase;
    int32_t op;
    int32_t dst;
    int32_t nsrc;
    int64_t src_off;  // index of the first source in Plan::srcs
    int64_t begin;
    int64_t end;
};

struct ExecState;  // device-side state, defined by the executor

struct Plan {
    int32_t n = 0;
    int64_t N = 0;
    int32_t dtype = 0;
    int32_t esize = 0;
    int32_t kind = -1;  // ar_kind, or -1 for custom plans
    std::vector<int32_t> fanin;
    std::vector<Step> steps;            // sorted by phase
    std::vector<int32_t> srcs;          // source pool
    std::vector<int64_t> phase_first;   // num_phases + 1 entries
    std::vector<int64_t> owner_begin;   // per processor (empty: unknown)
    std::vector<int64_t> owner_end;
    int32_t fuse = 1;   // AR_OPT_FUSE
    int32_t slice = 2;  // AR_OPT_SLICE: 0 never, 1 always (if possible), 2 auto
    int32_t resident = 1;  // AR_OPT_RESIDENT: sliced runs may keep their state in LDS
    ExecState* exec = nullptr;  // executor cache, built on first use

    int32_t num_phases() const {
        return phase_first.empty() ? 0 : int32_t(phase_first.size() - 1);
    }
    void add(int32_t phase, int32_t op, int32_t dst,
             const std::vector<int32_t>& s, int64_t b, int64_t e);
    void finish_phases();  // fills phase_first (steps already in order)
};

// Element offset of block b of the n-way split of N elements: the floor
// share each, one more for each of the first N mod n blocks.
inline int64_t block_off(int64_t N, int32_t n, int64_t b) {
    const int64_t q = N / n, r = N % n;
    return b * q + (b < r ? b : r);
}

// Expanders; they throw std::invalid_argument / arp::Unsupported.
struct Unsupported : std::exception {
    std::string msg;
    explicit Unsupported(std::string m) : msg(std::move(m)) {}
    const char* what() const noexcept override { return msg.c_str(); }
};

void expand_ring(Plan& p);
void expand_rhd(Plan& p);
void expand_cps(Plan& p);
void expand_tree(Plan& p);  // uses p.fanin
void expand_rb(Plan& p);
// GenTree basic plan on an arbitrary tree given as child counts in
// preorder (0 = server); p.n must already be the number of servers.
void expand_gentree(Plan& p, const std::vector<int32_t>& nchild);
// Number of servers of a preorder child-count list, or -1 if the list does
// not describe exactly one tree.
int64_t gentree_servers(const std::vector<int32_t>& nchild);

// Throws std::invalid_argument naming the first hazard found.
void validate_phases(const Plan& p);

int64_t step_bytes(const Plan& p, const Step& s);

}  // namespace arp
