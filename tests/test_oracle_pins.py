"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: the
element-wise sum (brute force, exact in int32 and for small integers in
fp32), textbook folds in the order the paper describes, closed-form step
and byte counts of Tables 1-2 and Theorem 1, the GenModel term proportions
printed for Figure 8, the placement rule of Algorithm 1, and bf16 rounding
of a library routine.
"""

import functools
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import model
from paper_2409_04202_amd import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# -- plan catalogue for tiny shapes ---------------------------------------

def _factorizations(n, maxlen=4):
    """Ordered factorizations of n into factors >= 2 (fan-in vectors)."""
    out = []

    def rec(rest, cur):
        if rest == 1:
            if cur:
                out.append(tuple(cur))
            return
        if len(cur) == maxlen:
            return
        for f in range(2, rest + 1):
            if rest % f == 0:
                rec(rest // f, cur + [f])
    rec(n, [])
    return out


def tiny_plans(n, N):
    plans = [oracle.ring(n, N), oracle.cps(n, N), oracle.reduce_broadcast(n, N),
             oracle.rhd(n, N)]
    for fan in _factorizations(n):
        if len(fan) > 1:
            plans.append(oracle.tree(fan, N))
    return plans


TINY_N = [1, 2, 3, 4, 5, 6, 7, 8, 9, 12, 16]


def tiny_sizes(n):
    return sorted({0, 1, max(n - 1, 0), n, 7, 33, 1000})


# -- P1: brute force ------------------------------------------------------

@pytest.mark.parametrize("n", TINY_N)
def test_int32_equals_elementwise_sum(n):
    for N in tiny_sizes(n):
        xs0 = workloads.draw(n, N, "i32", "int1000", 7 + n)
        ref = (np.sum([x.astype(np.int64) for x in xs0], axis=0)
               .astype(np.int32) if N else np.zeros(0, np.int32))
        for p in tiny_plans(n, N):
            xs = oracle.execute(p, [x.copy() for x in xs0], "i32")
            for q in range(n):
                assert np.array_equal(xs[q], ref), (p, q, N)


def test_int32_wraps_like_twos_complement():
    n, N = 4, 9
    big = np.iinfo(np.int32).max
    xs0 = [np.full(N, big, np.int32) for _ in range(n)]
    ref = ((np.int64(big) * n + 2**31) % 2**32 - 2**31).astype(np.int32)
    for p in tiny_plans(n, N):
        xs = oracle.execute(p, [x.copy() for x in xs0], "i32")
        assert all(np.all(x == ref) for x in xs), p


@pytest.mark.parametrize("n", TINY_N)
def test_fp32_small_integers_are_exact(n):
    # |x| <= 1000 integers: every partial sum is an integer below 2^24, so
    # fp32 is exact for every association order.
    for N in (n, 33):
        xs0 = workloads.draw(n, N, "f32", "smallint", 11 + n)
        ref = np.sum([x.astype(np.float64) for x in xs0], axis=0)
        for p in tiny_plans(n, N):
            xs = oracle.execute(p, [x.copy() for x in xs0], "f32")
            for q in range(n):
                assert np.array_equal(xs[q].astype(np.float64), ref), (p, q)


@pytest.mark.parametrize("n", [3, 8, 12, 16])
def test_fp32_random_within_summation_bound(n):
    # Any association order of n - 1 fp32 additions has error at most
    # gamma_{n-1} * sum|x|, gamma_k = k u / (1 - k u), u = 2^-24.
    N = 257
    xs0 = workloads.draw(n, N, "f32", "uniform", 5 + n)
    exact = np.sum([x.astype(np.float64) for x in xs0], axis=0)
    mag = np.sum([np.abs(x.astype(np.float64)) for x in xs0], axis=0)
    u = 2.0 ** -24
    gam = (n - 1) * u / (1 - (n - 1) * u)
    for p in tiny_plans(n, N):
        xs = oracle.execute(p, [x.copy() for x in xs0], "f32")
        err = np.abs(xs[0].astype(np.float64) - exact)
        assert np.all(err <= gam * mag), p


# -- P2: every input counted exactly once (symbolic counts) ---------------

@pytest.mark.parametrize("n", [2, 3, 4, 6, 8, 12])
def test_each_input_contributes_exactly_once(n):
    for N in (n, 2 * n + 3):
        for p in tiny_plans(n, N):
            # buffer q holds, per element, a count vector with a 1 at q
            xs = []
            for q in range(n):
                a = np.zeros((N, n), np.int64)
                a[:, q] = 1
                xs.append(a)
            oracle.execute(p, xs, "i32")
            for q in range(n):
                assert np.all(xs[q] == 1), (p, q)


# -- P3: invariants -------------------------------------------------------

def _sequential(plan, bufs, dtype, reverse):
    """Execute steps one at a time, in place (no phase snapshot)."""
    for ph in plan.phases:
        for st in (reversed(ph) if reverse else ph):
            if st.op == "reduce":
                val = oracle.fold(dtype, [bufs[s][st.begin:st.end]
                                          for s in st.srcs])
            else:
                val = bufs[st.srcs[0]][st.begin:st.end].copy()
            bufs[st.dst][st.begin:st.end] = val
    return bufs


@pytest.mark.parametrize("n", [2, 3, 4, 8, 12, 16])
def test_steps_of_a_phase_are_independent(n):
    # In-place execution in any step order equals the phase-snapshot
    # execution: no step reads or writes what another step of its phase
    # writes.
    N = 3 * n + 5
    xs0 = workloads.draw(n, N, "f32", "uniform", 3)
    for p in tiny_plans(n, N):
        ref = oracle.execute(p, [x.copy() for x in xs0], "f32")
        for rev in (False, True):
            got = _sequential(p, [x.copy() for x in xs0], "f32", rev)
            for q in range(n):
                assert np.array_equal(got[q], ref[q]), (p, rev)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_all_outputs_bitwise_identical(dtype):
    for n in (5, 8, 12, 16):
        N = 100
        xs0 = workloads.draw(n, N, dtype, "uniform", 9)
        for p in tiny_plans(n, N):
            xs = oracle.execute(p, [x.copy() for x in xs0], dtype)
            for q in range(1, n):
                assert np.array_equal(xs[q], xs[0]), (p, q)


def test_sampled_execution_equals_full():
    for name, n, fan in (("ring", 8, None), ("tree", 12, (3, 4)),
                         ("rhd", 8, None), ("cps", 6, None)):
        N = 1001
        p = oracle.make_plan(name, n, N, fan)
        xs0 = workloads.draw(n, N, "bf16", "uniform", 2)
        full = oracle.execute(p, [x.copy() for x in xs0], "bf16")
        idx = np.array([0, 1, 77, 500, 999, 1000])
        got = oracle.execute_sampled(p, [x[idx] for x in xs0], idx, "bf16")
        for q in range(n):
            assert np.array_equal(got[q], full[q][idx])


# -- P8: the association order the paper describes ------------------------

def test_cps_is_left_fold_in_rank_order():
    # a_0 + a_1 + ... + a_{n-1} (Section 3.1), as a textbook left fold.
    n, N = 16, 4099
    xs0 = workloads.draw(n, N, "f32", "normal", 21)
    ref = functools.reduce(lambda a, b: np.add(a, b, dtype=np.float32), xs0)
    xs = oracle.execute(oracle.cps(n, N), [x.copy() for x in xs0], "f32")
    assert np.array_equal(xs[5], ref)
    xs = oracle.execute(oracle.reduce_broadcast(n, N),
                        [x.copy() for x in xs0], "f32")
    assert np.array_equal(xs[0], ref)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ring_block_is_cyclic_fold(dtype):
    # Block b travels b-1 -> b -> b+1 -> ... -> b-2 (Section 2.1, Ring),
    # each hop adding the local value; bf16 rounds after each hop.
    n, N = 7, 7 * 13 + 4
    xs0 = workloads.draw(n, N, dtype, "uniform", 31)
    xs = oracle.execute(oracle.ring(n, N), [x.copy() for x in xs0], dtype)
    off = oracle.block_bounds(N, n)
    wid = oracle.bf16_to_f32
    for b in range(n):
        sl = slice(off[b], off[b + 1])
        order = [(b - 1 + t) % n for t in range(n)]
        acc = xs0[order[0]][sl]
        for q in order[1:]:
            if dtype == "f32":
                acc = np.add(acc, xs0[q][sl], dtype=np.float32)
            else:
                s = np.add(wid(acc), wid(xs0[q][sl]), dtype=np.float32)
                acc = torch.from_numpy(s).to(torch.bfloat16).view(
                    torch.int16).numpy().view(np.uint16)
        assert np.array_equal(xs[0][sl], acc), b


@pytest.mark.parametrize("fan,dtype", [((3, 4), "f32"), ((4, 3), "f32"),
                                       ((2, 3, 2), "f32"), ((8, 8), "bf16"),
                                       ((4, 2, 2), "bf16")])
def test_tree_is_nested_group_fold(fan, dtype):
    # Hierarchical CPS (Section 3.3): groups of f_0 consecutive ranks sum
    # first, then orthogonal groups of f_1, ...; each group sum is a left
    # fold in rank order, rounded once to bf16 per level.
    n = int(np.prod(fan))
    N = 5 * n + 3
    xs0 = workloads.draw(n, N, dtype, "uniform", 41)
    got = oracle.execute(oracle.tree(fan, N), [x.copy() for x in xs0], dtype)
    X = np.stack(xs0).reshape(tuple(reversed(fan)) + (N,))
    for lvl in range(len(fan)):
        axis = X.ndim - 2          # the fastest-varying remaining digit
        parts = [np.take(X, a, axis=axis) for a in range(X.shape[axis])]
        if dtype == "f32":
            X = functools.reduce(lambda a, b: np.add(a, b, dtype=np.float32),
                                 parts)
        else:
            f = functools.reduce(
                lambda a, b: np.add(a, b, dtype=np.float32),
                [oracle.bf16_to_f32(t) for t in parts])
            X = torch.from_numpy(np.ascontiguousarray(f)).to(
                torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(got[n - 1], X)


@pytest.mark.parametrize("k", [1, 2, 3, 4])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_rhd_equals_binary_tree(k, dtype):
    # Two independent expanders: nearest-partner-first RHD and the
    # hierarchical CPS with every fan-in 2.
    n = 2 ** k
    for N in (n, 10 * n + 3, 1):
        xs0 = workloads.draw(n, N, dtype, "uniform", 51)
        a = oracle.execute(oracle.rhd(n, N), [x.copy() for x in xs0], dtype)
        b = oracle.execute(oracle.tree((2,) * k, N), [x.copy() for x in xs0],
                           dtype)
        for q in range(n):
            assert np.array_equal(a[q], b[q])


@pytest.mark.parametrize("k", [1, 2, 3, 4])
def test_rhd_steps_equal_binary_tree_steps(k):
    # Same steps, hence the same owners: the tree's owners are pinned to
    # Algorithm 1, so this also fixes which half RHD keeps.
    n = 2 ** k
    for N in (n, 7 * n + 5):
        pa, pb = oracle.rhd(n, N), oracle.tree((2,) * k, N)
        assert len(pa.phases) == len(pb.phases)
        for a, b in zip(pa.phases, pb.phases):
            assert sorted(a) == sorted(b)


def test_cps_equals_single_level_tree():
    n, N = 12, 101
    pa, pb = oracle.cps(n, N), oracle.tree((n,), N)
    assert [sorted(ph) for ph in pa.phases] == [sorted(ph) for ph in pb.phases]


def test_two_processors_all_plans_agree():
    N = 77
    xs0 = workloads.draw(2, N, "f32", "uniform", 61)
    outs = [oracle.execute(p, [x.copy() for x in xs0], "f32")[0]
            for p in tiny_plans(2, N)]
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


def test_single_processor_is_identity():
    for p in tiny_plans(1, 10):
        assert p.phases == []
        x = np.arange(10, dtype=np.float32)
        assert np.array_equal(oracle.execute(p, [x.copy()], "f32")[0], x)


# -- P4: step counts of Section 2.1 / Tables 1-2 --------------------------

@pytest.mark.parametrize("n", [2, 3, 4, 5, 8, 12, 16])
def test_ring_steps_follow_section_2_1(n):
    N = 12 * n
    p = oracle.ring(n, N)
    assert len(p.phases) == 2 * (n - 1)
    off = oracle.block_bounds(N, n)
    for j, ph in enumerate(p.phases):
        assert len(ph) == n
        for st in ph:
            i = st.dst
            blk = (i - j) % n                 # receives block (i - j) % n
            assert (st.begin, st.end) == (off[blk], off[blk + 1])
            left = (i - 1) % n                # from the left neighbour
            assert left in st.srcs
            assert st.op == ("reduce" if j < n - 1 else "copy")


@pytest.mark.parametrize("k", [1, 2, 3, 4, 5])
def test_rhd_steps_follow_section_2_1(k):
    n = 2 ** k
    N = n * 64
    p = oracle.rhd(n, N)
    assert len(p.phases) == 2 * k
    for j in range(k):       # halving step j moves 2^-(j+1) of the data
        for st in p.phases[j]:
            assert st.end - st.begin == N >> (j + 1)
            assert st.op == "reduce" and len(st.srcs) == 2
            assert set(st.srcs) == {st.dst, st.dst ^ (1 << j)}
    for j in range(k):       # doubling mirrors them
        for st in p.phases[k + j]:
            assert st.end - st.begin == N >> (k - j)
            assert st.op == "copy"


def test_round_counts_table_1():
    # A coefficients: RB 2, CPS 2, Ring 2(n-1), RHD 2 ceil(log n), HCPS 2m.
    for n in (2, 3, 4, 5, 6, 7, 8, 12, 16, 17, 32):
        N = 4 * n
        assert model.num_phases(oracle.reduce_broadcast(n, N)) == 2
        assert model.num_phases(oracle.cps(n, N)) == 2
        assert model.num_phases(oracle.ring(n, N)) == 2 * (n - 1)
        assert model.num_phases(oracle.rhd(n, N)) == 2 * (n - 1).bit_length()
    for fan in ((8, 8), (8, 8, 8), (2, 6), (3, 2, 2)):
        assert model.num_phases(oracle.tree(fan, 1000)) == 2 * len(fan)


# -- P5: memory, computation and traffic counts (Table 2, Theorem 1) ------

def _hcps_delta_numerator(fan):
    # Theorem 1, eq. (mem3) applied to hierarchical CPS: per block,
    # h = sum over levels l of prod_{l' > l} f_l'; D = (n - 1 + 2h) S / n.
    n = int(np.prod(fan))
    h = sum(int(np.prod(fan[l + 1:])) for l in range(len(fan)))
    return n - 1 + 2 * h


@pytest.mark.parametrize("n", [2, 4, 8, 16])
def test_delta_gamma_beta_counts_tables_1_2(n):
    N = n * 24
    per = lambda x: x / n
    ring = oracle.ring(n, N)
    assert per(model.reduce_memory_ops(ring)) == 3 * (n - 1) * N / n
    rhd = oracle.rhd(n, N)
    assert per(model.reduce_memory_ops(rhd)) == 3 * (n - 1) * N / n
    cps = oracle.cps(n, N)
    assert per(model.reduce_memory_ops(cps)) == (n + 1) * N / n
    rb = oracle.reduce_broadcast(n, N)
    assert model.reduce_memory_ops(rb) == (n + 1) * N
    assert model.add_ops(rb) == (n - 1) * N
    for p in (ring, rhd, cps):
        assert per(model.add_ops(p)) == (n - 1) * N / n          # gamma
        # bandwidth-optimal traffic, eq. (bw_op): 2 (n-1) S / n each way
        assert model.received_elements(p) == [2 * (n - 1) * N // n] * n
        assert model.sent_elements(p) == [2 * (n - 1) * N // n] * n


@pytest.mark.parametrize("fan", [(2, 6), (6, 2), (3, 4), (4, 3), (8, 8),
                                 (8, 8, 8), (2, 3, 4), (4, 3, 2), (2, 2, 2, 2)])
def test_theorem_1_per_block(fan):
    n = int(np.prod(fan))
    N = 2 * n
    p = oracle.tree(fan, N)
    h_expected = sum(int(np.prod(fan[l + 1:])) for l in range(len(fan)))
    for b, fins in enumerate(model.block_fanins(p)):
        assert sum(f - 1 for f in fins) == n - 1          # eq. (mem1)
        assert len(fins) == h_expected
    # eq. (mem3): total memory operations
    assert model.reduce_memory_ops(p) == _hcps_delta_numerator(fan) * N
    # Table 2 prints 2 * sum_{i=1}^{m-1} prod_{j=1}^{i} f_j + n + 1; it
    # agrees with Theorem 1 for two levels and for equal fan-ins.
    m = len(fan)
    table2 = 2 * sum(int(np.prod(fan[1:i + 1])) for i in range(1, m)) + n + 1
    if m <= 2 or len(set(fan[1:])) == 1:
        assert model.reduce_memory_ops(p) == table2 * N
    assert model.received_elements(p) == [2 * (n - 1) * N // n] * n


def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _plan_12(name, fans):
    if name == "Ring":
        return oracle.ring(12, 1200)
    if name == "CPS":
        return oracle.cps(12, 1200)
    return oracle.tree(tuple(int(f) for f in fans.split(",")), 1200)


def test_genmodel_term_ratios_match_figure_8():
    # The bandwidth+computation term is the same for every plan, so the
    # ratios memory/bc and latency/bc are proportional to D and A.
    rows = _read_golden("fig8_genmodel_terms_12proc.txt")
    ref = {r[0]: r for r in rows}
    cps = oracle.cps(12, 1200)
    d_cps = model.reduce_memory_ops(cps)
    a_cps = model.num_phases(cps)
    r_cps = ref["CPS"]
    for name, fans, bc, _inc, mem, lat in rows:
        p = _plan_12(name, fans)
        want_d = (float(mem) / float(bc)) / (float(r_cps[4]) / float(r_cps[2]))
        got_d = model.reduce_memory_ops(p) / d_cps
        assert abs(got_d - want_d) < 1e-6 * want_d, (name, got_d, want_d)
        want_a = (float(lat) / float(bc)) / (float(r_cps[5]) / float(r_cps[2]))
        got_a = model.num_phases(p) / a_cps
        assert abs(got_a - want_a) < 1e-6 * want_a, (name, got_a, want_a)


def test_memory_counts_track_measured_calc_time_figure_7():
    # Measured reduce time on the CPU testbed (10 Gbps) relative to CPS
    # follows the delta coefficient within 5 %.
    rows = _read_golden("fig7_calc_time_12proc.txt")
    t_cps = float([r for r in rows if r[0] == "CPS"][0][2])
    d_cps = model.reduce_memory_ops(oracle.cps(12, 1200))
    for name, fans, t10, _t100 in rows:
        p = _plan_12(name, fans)
        ratio_model = model.reduce_memory_ops(p) / d_cps
        ratio_meas = float(t10) / t_cps
        assert abs(ratio_meas / ratio_model - 1) < 0.05, name


# -- P6: Algorithm 1 placement -------------------------------------------

@pytest.mark.parametrize("fan", [(2,), (5,), (3, 2), (2, 3), (8, 8),
                                 (2, 2, 2), (8, 8, 8), (2, 3, 4)])
def test_tree_ownership_matches_algorithm_1(fan):
    n = int(np.prod(fan))
    N = n   # one element per block: ranges are block indices
    p = oracle.tree(fan, N)
    root = oracle.symmetric_tree(fan)
    place = oracle.basic_placement(root, n)
    levels = oracle.gentree.switch_levels(root)
    for l, switches in enumerate(levels):
        rs = p.phases[l]
        owned = {st.dst: list(range(st.begin, st.end)) for st in rs}
        for sw in switches:
            for sid, blocks in place[id(sw)].items():
                assert owned[sid] == blocks, (fan, l, sid)


def test_algorithm_1_on_an_asymmetric_tree():
    # Hand-checked: switch A has 2 servers, switch B has 3; root above.
    # With n = 5 blocks, A's servers take {0,1,2} and {3,4}; B's take
    # {0,1},{2,3},{4}; at the root the five servers take one block each,
    # first untaken in their own order.
    root = oracle.switch([oracle.switch([oracle.server(), oracle.server()]),
                          oracle.switch([oracle.server(), oracle.server(),
                                         oracle.server()])])
    oracle.gentree.number_servers(root)
    place = oracle.basic_placement(root, 5)
    a, b = root.children
    assert place[id(a)] == {0: [0, 1, 2], 1: [3, 4]}
    assert place[id(b)] == {2: [0, 1], 3: [2, 3], 4: [4]}
    assert place[id(root)] == {0: [0], 1: [3], 2: [1], 3: [2], 4: [4]}


# -- P9: bf16 rounding ----------------------------------------------------

def test_bf16_round_to_nearest_even_matches_torch():
    rng = np.random.default_rng(0)
    vals = [rng.standard_normal(100000).astype(np.float32),
            (rng.random(10000, dtype=np.float32) * 2 - 1) * np.float32(1e-38)]
    # exact ties: low 16 bits = 0x8000 with even and odd kept parts
    hi = rng.integers(0, 0x7F7F, size=5000).astype(np.uint32)
    for low in (0x8000, 0x7FFF, 0x8001, 0x0000, 0xFFFF):
        vals.append(((hi << 16) | low).view(np.float32))
        vals.append((((hi << 16) | low) | np.uint32(0x80000000))
                    .view(np.float32))
    vals.append(np.array([0.0, -0.0, np.inf, -np.inf, 3.3895314e38,
                          3.4028235e38, 1e-45, -1e-45], np.float32))
    for v in vals:
        got = oracle.f32_to_bf16(v)
        want = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16) \
                    .numpy().view(np.uint16)
        assert np.array_equal(got, want)
    b = np.arange(0, 65536, dtype=np.uint16)
    f = oracle.bf16_to_f32(b)
    finite = ~np.isnan(f)
    assert np.array_equal(oracle.f32_to_bf16(f)[finite], b[finite])


def test_block_bounds_floor_plus_remainder():
    assert oracle.block_bounds(10, 4) == [0, 3, 6, 8, 10]
    assert oracle.block_bounds(3, 5) == [0, 1, 2, 3, 3, 3]
    assert oracle.block_bounds(0, 3) == [0, 0, 0, 0]


@pytest.mark.parametrize("n", [3, 5, 6, 7, 12, 17])
def test_rhd_non_power_of_two_extra_terms(n):
    # Tables 1 and 2: with chi(n) = 1 the plan costs 2S beta + S gamma +
    # 3S delta more than the power-of-two part, on the processor that takes
    # an extra one in; the inner part is exactly RHD on the first p ranks.
    N = 8 * n + 3
    p = 1 << (n.bit_length() - 1)
    full = oracle.rhd(n, N)
    inner = oracle.rhd(p, N)
    assert full.phases[1:-1] == inner.phases
    pre, post = full.phases[0], full.phases[-1]
    assert all(st.op == "reduce" and (st.begin, st.end) == (0, N) for st in pre)
    assert all(st.op == "copy" and (st.begin, st.end) == (0, N) for st in post)
    assert sorted(st.dst for st in pre) == list(range(n - p))
    mem = lambda plan, r: sum((len(s.srcs) + 1) * (s.end - s.begin)
                              for s in plan.steps if s.op == "reduce" and s.dst == r)
    adds = lambda plan, r: sum((len(s.srcs) - 1) * (s.end - s.begin)
                               for s in plan.steps if s.op == "reduce" and s.dst == r)
    for r in range(n - p):      # processors that take an extra one in
        assert mem(full, r) - mem(inner, r) == 3 * N          # 3S delta
        assert adds(full, r) - adds(inner, r) == N            # S gamma
    for q in range(p, n):       # the extra processors: S out, S back in
        assert model.sent_elements(full)[q] == N
        assert model.received_elements(full)[q] == N
