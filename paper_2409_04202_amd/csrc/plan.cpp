// Plan expanders and the phase hazard check (host only, no HIP).
//
// Plan definitions follow Section 2.1 (Ring, RHD, co-located PS,
// Reduce-Broadcast), Section 3.3 (hierarchical co-located PS) and the
// bottom-up block placement of Algorithm 1; the exact rules are stated
// with each kind in include/ar_plan.h.
#include "plan.hpp"

#include <algorithm>
#include <stdexcept>

namespace arp {

void Plan::add(int32_t phase, int32_t op, int32_t dst,
               const std::vector<int32_t>& s, int64_t b, int64_t e) {
    Step st;
    st.phase = phase;
    st.op = op;
    st.dst = dst;
    st.nsrc = int32_t(s.size());
    st.src_off = int64_t(srcs.size());
    st.begin = b;
    st.end = e;
    srcs.insert(srcs.end(), s.begin(), s.end());
    steps.push_back(st);
}

void Plan::finish_phases() {
    phase_first.clear();
    int32_t nph = steps.empty() ? 0 : steps.back().phase + 1;
    phase_first.assign(size_t(nph) + 1, int64_t(steps.size()));
    for (int64_t i = int64_t(steps.size()) - 1; i >= 0; --i)
        phase_first[size_t(steps[size_t(i)].phase)] = i;
    for (int32_t ph = nph - 1; ph >= 0; --ph)  // phases without steps
        if (phase_first[size_t(ph)] > phase_first[size_t(ph) + 1])
            phase_first[size_t(ph)] = phase_first[size_t(ph) + 1];
}

static inline int32_t pmod(int64_t a, int32_t n) {
    int64_t r = a % n;
    return int32_t(r < 0 ? r + n : r);
}

// Ring: in step j processor i receives block (i - j) mod n from i - 1.
void expand_ring(Plan& p) {
    const int32_t n = p.n;
    const int64_t N = p.N;
    p.owner_begin.assign(size_t(n), 0);
    p.owner_end.assign(size_t(n), N);
    if (n == 1) { p.finish_phases(); return; }
    for (int32_t j = 0; j < 2 * (n - 1); ++j) {
        for (int32_t i = 0; i < n; ++i) {
            const int32_t b = pmod(int64_t(i) - j, n);
            const int32_t left = pmod(int64_t(i) - 1, n);
            const int64_t lo = block_off(N, n, b), hi = block_off(N, n, b + 1);
            if (j < n - 1)
                p.add(j, OP_REDUCE, i, {i, left}, lo, hi);
            else
                p.add(j, OP_COPY, i, {left}, lo, hi);
        }
    }
    for (int32_t i = 0; i < n; ++i) {  // block reduced in step n - 2
        const int32_t b = pmod(int64_t(i) + 2, n);
        p.owner_begin[size_t(i)] = block_off(N, n, b);
        p.owner_end[size_t(i)] = block_off(N, n, b + 1);
    }
    p.finish_phases();
}

// Recursive halving-doubling, nearest partner (r XOR 1) first; r keeps the
// lower half when bit j of r is 0.  For n not a power of two, with p the
// largest power of two below n: processor q >= p first reduces its whole
// buffer into q - p, the first p processors run the power-of-two plan, and
// q copies the result back from q - p (the two extra steps).
static void rhd_pow2(Plan& p, int32_t n, int32_t ph0);

void expand_rhd(Plan& p) {
    const int32_t n = p.n;
    const int64_t N = p.N;
    if (n & (n - 1)) {
        int32_t pw = 1;
        while (pw * 2 <= n) pw *= 2;
        for (int32_t q = pw; q < n; ++q) p.add(0, OP_REDUCE, q - pw, {q - pw, q}, 0, N);
        rhd_pow2(p, pw, 1);
        const int32_t last = p.steps.empty() ? 1 : p.steps.back().phase + 1;
        for (int32_t q = pw; q < n; ++q) p.add(last, OP_COPY, q, {q - pw}, 0, N);
        // owners: the power-of-two part as computed; the extra ones own nothing
        for (int32_t q = pw; q < n; ++q) {
            p.owner_begin[size_t(q)] = 0;
            p.owner_end[size_t(q)] = 0;
        }
        p.finish_phases();
        return;
    }
    rhd_pow2(p, n, 0);
    p.finish_phases();
}

static void rhd_pow2(Plan& p, int32_t n, int32_t ph0) {
    const int64_t N = p.N;
    int32_t k = 0;
    while ((1 << k) < n) ++k;
    std::vector<std::pair<int32_t, int32_t>> held(size_t(n), {0, n});
    std::vector<std::vector<std::pair<int32_t, int32_t>>> kept;
    for (int32_t j = 0; j < k; ++j) {
        std::vector<std::pair<int32_t, int32_t>> nk(static_cast<size_t>(n));
        for (int32_t r = 0; r < n; ++r) {
            const auto [lo, hi] = held[size_t(r)];
            const int32_t mid = (lo + hi) / 2;
            nk[size_t(r)] = ((r >> j) & 1) ? std::make_pair(mid, hi)
                                           : std::make_pair(lo, mid);
            const int32_t q = r ^ (1 << j);
            p.add(ph0 + j, OP_REDUCE, r, {std::min(r, q), std::max(r, q)},
                  block_off(N, n, nk[size_t(r)].first),
                  block_off(N, n, nk[size_t(r)].second));
        }
        held = nk;
        kept.push_back(nk);
    }
    for (int32_t jj = 0; jj < k; ++jj) {
        const int32_t j = k - 1 - jj;
        for (int32_t r = 0; r < n; ++r) {
            const int32_t q = r ^ (1 << j);
            const auto [lo, hi] = kept[size_t(j)][size_t(q)];
            p.add(ph0 + k + jj, OP_COPY, r, {q}, block_off(N, n, lo),
                  block_off(N, n, hi));
        }
    }
    p.owner_begin.resize(size_t(p.n));
    p.owner_end.resize(size_t(p.n));
    for (int32_t r = 0; r < n; ++r) {
        p.owner_begin[size_t(r)] = block_off(N, n, held[size_t(r)].first);
        p.owner_end[size_t(r)] = block_off(N, n, held[size_t(r)].second);
    }
}

// Co-located PS: one n-way reduce per block, then n - 1 copies per block.
void expand_cps(Plan& p) {
    const int32_t n = p.n;
    const int64_t N = p.N;
    p.owner_begin.resize(size_t(n));
    p.owner_end.resize(size_t(n));
    for (int32_t r = 0; r < n; ++r) {
        p.owner_begin[size_t(r)] = block_off(N, n, r);
        p.owner_end[size_t(r)] = block_off(N, n, r + 1);
    }
    if (n == 1) { p.finish_phases(); return; }
    std::vector<int32_t> all(static_cast<size_t>(n));
    for (int32_t r = 0; r < n; ++r) all[size_t(r)] = r;
    for (int32_t r = 0; r < n; ++r)
        p.add(0, OP_REDUCE, r, all, block_off(N, n, r), block_off(N, n, r + 1));
    for (int32_t r = 0; r < n; ++r)
        for (int32_t q = 0; q < n; ++q)
            if (q != r)
                p.add(1, OP_COPY, r, {q}, block_off(N, n, q),
                      block_off(N, n, q + 1));
    p.finish_phases();
}

// Hierarchical co-located PS over fan-ins f_0 (innermost) .. f_{m-1}.
void expand_tree(Plan& p) {
    const int32_t n = p.n;
    const int64_t N = p.N;
    const int32_t m = int32_t(p.fanin.size());
    std::vector<int64_t> stride(static_cast<size_t>(m)), prod(static_cast<size_t>(m));
    int64_t s = 1;
    for (int32_t l = 0; l < m; ++l) {
        stride[size_t(l)] = s;
        s *= p.fanin[size_t(l)];
        prod[size_t(l)] = s;
    }
    if (s != n) throw std::invalid_argument("product of fan-ins != n");
    auto digit = [&](int32_t r, int32_t l) {
        return int32_t((r / stride[size_t(l)]) % p.fanin[size_t(l)]);
    };
    // own_lo[l][r]: first block owned by r after level l (width n / prod[l])
    std::vector<std::vector<int64_t>> own_lo(static_cast<size_t>(m),
                                             std::vector<int64_t>(static_cast<size_t>(n)));
    std::vector<int64_t> o(size_t(n), 0);
    for (int32_t l = 0; l < m; ++l) {
        const int64_t width = n / prod[size_t(l)];
        for (int32_t r = 0; r < n; ++r) {
            o[size_t(r)] = o[size_t(r)] * p.fanin[size_t(l)] + digit(r, l);
            own_lo[size_t(l)][size_t(r)] = o[size_t(r)] * width;
        }
    }
    auto group = [&](int32_t r, int32_t l) {
        std::vector<int32_t> g(static_cast<size_t>(p.fanin[size_t(l)]));
        const int32_t d = digit(r, l);
        for (int32_t a = 0; a < p.fanin[size_t(l)]; ++a)
            g[size_t(a)] = int32_t(r + (int64_t(a) - d) * stride[size_t(l)]);
        return g;
    };
    auto range = [&](int32_t l, int32_t r) {
        const int64_t width = n / prod[size_t(l)];
        const int64_t lo = own_lo[size_t(l)][size_t(r)];
        return std::make_pair(block_off(N, n, lo), block_off(N, n, lo + width));
    };
    int32_t ph = 0;
    for (int32_t l = 0; l < m; ++l) {
        if (p.fanin[size_t(l)] == 1) continue;
        for (int32_t r = 0; r < n; ++r) {
            const auto [b, e] = range(l, r);
            p.add(ph, OP_REDUCE, r, group(r, l), b, e);
        }
        ++ph;
    }
    for (int32_t l = m - 1; l >= 0; --l) {
        if (p.fanin[size_t(l)] == 1) continue;
        for (int32_t r = 0; r < n; ++r) {
            for (int32_t q : group(r, l)) {
                if (q == r) continue;
                const auto [b, e] = range(l, q);
                p.add(ph, OP_COPY, r, {q}, b, e);
            }
        }
        ++ph;
    }
    p.owner_begin.resize(size_t(n));
    p.owner_end.resize(size_t(n));
    for (int32_t r = 0; r < n; ++r) {
        if (m == 0) {
            p.owner_begin[size_t(r)] = 0;
            p.owner_end[size_t(r)] = N;
        } else {
            const auto [b, e] = range(m - 1, r);
            p.owner_begin[size_t(r)] = b;
            p.owner_end[size_t(r)] = e;
        }
    }
    p.finish_phases();
}

// Reduce-Broadcast: rank 0 reduces everything, then everyone copies it.
void expand_rb(Plan& p) {
    const int32_t n = p.n;
    const int64_t N = p.N;
    p.owner_begin.assign(size_t(n), 0);
    p.owner_end.assign(size_t(n), 0);
    p.owner_end[0] = N;
    if (n == 1) { p.finish_phases(); return; }
    std::vector<int32_t> all(static_cast<size_t>(n));
    for (int32_t r = 0; r < n; ++r) all[size_t(r)] = r;
    p.add(0, OP_REDUCE, 0, all, 0, N);
    for (int32_t r = 1; r < n; ++r) p.add(1, OP_COPY, r, {0}, 0, N);
    p.finish_phases();
}

int64_t step_bytes(const Plan& p, const Step& s) {
    const int64_t len = s.end - s.begin;
    const int64_t k = s.op == OP_COPY ? 1 : s.nsrc;
    return (k + 1) * len * p.esize;
}

namespace {
struct Iv {
    int32_t buf;
    int64_t b, e;
    int64_t step;
};
}  // namespace

void validate_phases(const Plan& p) {
    for (int32_t ph = 0; ph < p.num_phases(); ++ph) {
        const int64_t s0 = p.phase_first[size_t(ph)];
        const int64_t s1 = p.phase_first[size_t(ph) + 1];
        std::vector<Iv> w;
        w.reserve(size_t(s1 - s0));
        for (int64_t i = s0; i < s1; ++i) {
            const Step& st = p.steps[size_t(i)];
            if (st.end > st.begin) w.push_back({st.dst, st.begin, st.end, i});
        }
        std::sort(w.begin(), w.end(), [](const Iv& a, const Iv& b) {
            return a.buf != b.buf ? a.buf < b.buf : a.b < b.b;
        });
        for (size_t i = 1; i < w.size(); ++i)
            if (w[i].buf == w[i - 1].buf && w[i].b < w[i - 1].e)
                throw std::invalid_argument(
                    "phase " + std::to_string(ph) + ": steps " +
                    std::to_string(w[i - 1].step) + " and " +
                    std::to_string(w[i].step) + " write overlapping ranges");
        // reads must not overlap another step's write
        for (int64_t i = s0; i < s1; ++i) {
            const Step& st = p.steps[size_t(i)];
            if (st.end <= st.begin) continue;
            for (int32_t t = 0; t < st.nsrc; ++t) {
                const int32_t buf = p.srcs[size_t(st.src_off + t)];
                // first write on `buf` whose end is past st.begin
                auto it = std::lower_bound(
                    w.begin(), w.end(), std::make_pair(buf, st.begin),
                    [](const Iv& a, const std::pair<int32_t, int64_t>& key) {
                        return a.buf != key.first ? a.buf < key.first
                                                  : a.e <= key.second;
                    });
                for (; it != w.end() && it->buf == buf && it->b < st.end; ++it)
                    if (it->step != i)
                        throw std::invalid_argument(
                            "phase " + std::to_string(ph) + ": step " +
                            std::to_string(i) + " reads a range that step " +
                            std::to_string(it->step) + " writes");
            }
        }
    }
}

// ---------------------------------------------------------------- GenTree

int64_t gentree_servers(const std::vector<int32_t>& nchild) {
    // preorder: every node consumes its children; the list must end exactly
    // when the root is complete
    int64_t open = 1, servers = 0;
    for (size_t i = 0; i < nchild.size(); ++i) {
        if (open == 0 || nchild[i] < 0) return -1;
        --open;
        if (nchild[i] == 0) ++servers;
        open += nchild[i];
    }
    return open == 0 ? servers : -1;
}

namespace {

struct TNode {
    std::vector<int32_t> kids;  // node indices
    int32_t server = -1;        // server id for leaves
    int32_t height = 0;         // 0 for servers
    // placement after this node's ReduceScatter: servers in order, each
    // with its blocks in the order taken (leaves: every block, implicit)
    std::vector<std::pair<int32_t, std::vector<int32_t>>> place;
};

}  // namespace

// GenTree's basic plan on a tree given by preorder child counts.  Block
// placement (Algorithm 1), bottom-up: at a switch the servers below it, in
// child order, get quotas of floor(n / s) blocks, one more for the first
// n mod s, and claim in that order the first unclaimed blocks of what they
// held below their child; a block left unclaimed goes to its holder in the
// first child.  Each switch reduces every block over one holder per child
// (on children with unequal shares this is Section 4.2's asymmetric CPS:
// every partial goes straight to the block's new owner); switches of one
// height share a phase; the AllGather reverses it.
void expand_gentree(Plan& p, const std::vector<int32_t>& nchild) {
    const int32_t n = p.n;
    const int64_t N = p.N;
    const int32_t nn = int32_t(nchild.size());
    std::vector<TNode> t(static_cast<size_t>(nn));
    {   // build the tree from the preorder child counts
        std::vector<std::pair<int32_t, int32_t>> stack;  // (node, kids still to attach)
        int32_t sid = 0;
        for (int32_t i = 0; i < nn; ++i) {
            if (!stack.empty()) {
                t[size_t(stack.back().first)].kids.push_back(i);
                if (--stack.back().second == 0) stack.pop_back();
            }
            if (nchild[size_t(i)] == 0)
                t[size_t(i)].server = sid++;
            else
                stack.push_back({i, nchild[size_t(i)]});
            while (!stack.empty() && stack.back().second == 0) stack.pop_back();
        }
        if (sid != n) throw std::invalid_argument("server count differs from n");
    }
    // post-order (children before parents)
    std::vector<int32_t> order;
    {
        std::vector<std::pair<int32_t, size_t>> st{{0, 0}};
        while (!st.empty()) {
            auto& [v, k] = st.back();
            if (k < t[size_t(v)].kids.size()) {
                const int32_t c = t[size_t(v)].kids[k++];
                st.push_back({c, 0});
            } else {
                order.push_back(v);
                st.pop_back();
            }
        }
    }
    int32_t H = 0;
    for (int32_t v : order) {
        TNode& a = t[size_t(v)];
        if (a.server >= 0) continue;
        for (int32_t c : a.kids) a.height = std::max(a.height, t[size_t(c)].height + 1);
        H = std::max(H, a.height);
    }
    std::vector<std::vector<Step>> rs(static_cast<size_t>(H)), ag(static_cast<size_t>(H));
    std::vector<std::vector<int32_t>> rs_srcs(static_cast<size_t>(H)), ag_srcs(static_cast<size_t>(H));
    // next_free[b]: smallest unclaimed block >= b (path-halving union-find),
    // so that a member whose candidates are every block claims its share in
    // amortised constant time per block
    std::vector<int32_t> claimed(static_cast<size_t>(n)), next_free(static_cast<size_t>(n) + 1);
    auto find_free = [&](int32_t b) {
        while (next_free[size_t(b)] != b) {
            next_free[size_t(b)] = next_free[size_t(next_free[size_t(b)])];
            b = next_free[size_t(b)];
        }
        return b;
    };
    auto claim = [&](int32_t b) {
        claimed[size_t(b)] = 1;
        next_free[size_t(b)] = b + 1;
    };
    std::vector<int32_t> slot_of(static_cast<size_t>(n), -1);  // server -> index in place
    for (int32_t v : order) {
        TNode& a = t[size_t(v)];
        if (a.server >= 0) {
            a.place.push_back({a.server, {}});  // implicit: every block
            continue;
        }
        // The members of this switch: the servers below it in child order,
        // each with its candidate blocks (what it held below its child; a
        // server child: every block, in order), and their quotas, fixed up
        // front: floor(n / s) each, one more for the first n mod s.
        struct Member {
            int32_t sid;
            const std::vector<int32_t>* cands;  // nullptr: every block
        };
        const size_t nk = a.kids.size();
        std::vector<Member> members;
        for (size_t i = 0; i < nk; ++i) {
            const TNode& c = t[size_t(a.kids[i])];
            if (c.server >= 0) {
                members.push_back({c.server, nullptr});
            } else {
                for (const auto& pr : c.place) members.push_back({pr.first, &pr.second});
            }
        }
        const int64_t s = int64_t(members.size());
        std::vector<int64_t> quota(members.size(), n / s);
        for (int64_t j = 0; j < n % s; ++j) ++quota[size_t(j)];
        // holder of block b below child i: a server child holds every
        // block; a switch child's placement names the server
        std::vector<int32_t> const_holder(nk, -1);
        std::vector<std::vector<int32_t>> holders(nk);
        for (size_t i = 0; i < nk; ++i) {
            const TNode& c = t[size_t(a.kids[i])];
            if (c.server >= 0) {
                const_holder[i] = c.server;
            } else {
                holders[i].assign(size_t(n), -1);
                for (const auto& pr : c.place)
                    for (int32_t b : pr.second) holders[i][size_t(b)] = pr.first;
            }
        }
        auto holder = [&](size_t i, int32_t b) {
            return const_holder[i] >= 0 ? const_holder[i] : holders[i][size_t(b)];
        };
        // one claiming pass over the members in order
        std::fill(claimed.begin(), claimed.end(), 0);
        for (int32_t b = 0; b <= n; ++b) next_free[size_t(b)] = b;
        a.place.reserve(members.size());
        for (size_t j = 0; j < members.size(); ++j) {
            std::vector<int32_t> got;
            const size_t q = size_t(quota[j]);
            if (!members[j].cands) {
                for (int32_t b = find_free(0); got.size() < q && b < n; b = find_free(b)) {
                    claim(b);
                    got.push_back(b);
                }
            } else {
                for (auto it = members[j].cands->begin();
                     got.size() < q && it != members[j].cands->end(); ++it)
                    if (!claimed[size_t(*it)]) {
                        claim(*it);
                        got.push_back(*it);
                    }
            }
            slot_of[size_t(members[j].sid)] = int32_t(a.place.size());
            a.place.push_back({members[j].sid, std::move(got)});
        }
        // completion: an unclaimed block, in block order, joins the list of
        // its holder in the first child that holds it
        for (int32_t b = find_free(0); b < n; b = find_free(b)) {
            int32_t h = -1;
            for (size_t i = 0; i < nk && h < 0; ++i) h = holder(i, b);
            if (h < 0 || slot_of[size_t(h)] < 0) throw std::logic_error("block without holder");
            a.place[size_t(slot_of[size_t(h)])].second.push_back(b);
            claim(b);
        }
        // steps: runs of consecutive blocks of one server with equal holders
        const size_t lvl = size_t(a.height - 1);
        for (const auto& [sid, blocks] : a.place) {
            size_t i0 = 0;
            while (i0 < blocks.size()) {
                size_t i1 = i0 + 1;
                auto same = [&](int32_t x, int32_t y) {
                    for (size_t k = 0; k < nk; ++k)
                        if (holder(k, x) != holder(k, y)) return false;
                    return true;
                };
                while (i1 < blocks.size() && blocks[i1] == blocks[i1 - 1] + 1 &&
                       same(blocks[i1], blocks[i0]))
                    ++i1;
                const int32_t b0 = blocks[i0], b1 = blocks[i1 - 1];
                std::vector<int32_t> hs;
                for (size_t k = 0; k < nk; ++k) hs.push_back(holder(k, b0));
                if (!(hs.size() == 1 && hs[0] == sid)) {
                    const int64_t lo = block_off(N, n, b0), hi = block_off(N, n, int64_t(b1) + 1);
                    Step st{};
                    st.op = OP_REDUCE;
                    st.dst = sid;
                    st.nsrc = int32_t(hs.size());
                    st.src_off = int64_t(rs_srcs[lvl].size());
                    st.begin = lo;
                    st.end = hi;
                    rs_srcs[lvl].insert(rs_srcs[lvl].end(), hs.begin(), hs.end());
                    rs[lvl].push_back(st);
                    for (int32_t q : hs) {
                        if (q == sid) continue;
                        Step c{};
                        c.op = OP_COPY;
                        c.dst = q;
                        c.nsrc = 1;
                        c.src_off = int64_t(ag_srcs[lvl].size());
                        c.begin = lo;
                        c.end = hi;
                        ag_srcs[lvl].push_back(sid);
                        ag[lvl].push_back(c);
                    }
                }
                i0 = i1;
            }
        }
        // children's placements are no longer needed
        for (int32_t c : a.kids)
            if (t[size_t(c)].server < 0) t[size_t(c)].place.clear();
    }
    // phases: ReduceScatter by increasing height, AllGather by decreasing
    int32_t ph = 0;
    auto emit = [&](std::vector<Step>& steps, std::vector<int32_t>& pool) {
        if (steps.empty()) return;
        for (Step st : steps) {
            p.add(ph, st.op, st.dst,
                  std::vector<int32_t>(pool.begin() + st.src_off,
                                       pool.begin() + st.src_off + st.nsrc),
                  st.begin, st.end);
        }
        ++ph;
    };
    for (int32_t h = 0; h < H; ++h) emit(rs[size_t(h)], rs_srcs[size_t(h)]);
    for (int32_t h = H - 1; h >= 0; --h) emit(ag[size_t(h)], ag_srcs[size_t(h)]);
    // owner after the last ReduceScatter level: the root's placement
    p.owner_begin.assign(size_t(n), -1);
    p.owner_end.assign(size_t(n), -1);
    if (t[0].server >= 0) {
        p.owner_begin[0] = 0;
        p.owner_end[0] = N;
    } else {
        for (const auto& [sid, blocks] : t[0].place) {
            std::vector<int32_t> b = blocks;
            std::sort(b.begin(), b.end());
            bool contiguous = true;
            for (size_t i = 1; i < b.size(); ++i) contiguous = contiguous && b[i] == b[i - 1] + 1;
            if (b.empty()) {
                p.owner_begin[size_t(sid)] = p.owner_end[size_t(sid)] = 0;
            } else if (contiguous) {
                p.owner_begin[size_t(sid)] = block_off(N, n, b.front());
                p.owner_end[size_t(sid)] = block_off(N, n, int64_t(b.back()) + 1);
            }
        }
    }
    p.finish_phases();
}

}  // namespace arp
