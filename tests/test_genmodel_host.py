"""Host-side checks of the single-GPU GenModel fit (features, least squares,
plan selection).  No GPU: plans are created and inspected on the host only.

The features the library reports are checked against the oracle's own counts
of the same plans (rounds, and the delta / copy byte terms of Table 2), which
the oracle pins separately against Table 1 and Table 2.
"""

import numpy as np
import pytest

import oracle
from oracle import model

from paper_2409_04202_amd import arplan, genmodel


PLANS = [("ring", n, None) for n in (2, 3, 5, 8)] + \
        [("rhd", n, None) for n in (2, 6, 8, 12)] + \
        [("cps", n, None) for n in (2, 7, 16)] + \
        [("tree", 16, (4, 4)), ("tree", 24, (2, 3, 4)), ("tree", 12, (3, 4))]


@pytest.mark.parametrize("kind,n,fan", PLANS)
@pytest.mark.parametrize("N", [1, 1000, 4099])
def test_features_match_oracle_counts(kind, n, fan, N):
    ref = oracle.make_plan(kind, n, N, fan)
    with arplan.Plan(n, N, "f32", kind, fan) as p:
        A, D, B = genmodel.features(p)
    assert A == model.num_phases(ref)
    assert (D, B) == model.algorithmic_bytes(ref, 4)


def test_features_bf16_halve_bytes():
    with arplan.Plan(8, 4096, "f32", "ring") as p32, \
            arplan.Plan(8, 4096, "bf16", "ring") as p16:
        a32, a16 = genmodel.features(p32), genmodel.features(p16)
    assert a32[0] == a16[0]
    assert a32[1] == 2 * a16[1] and a32[2] == 2 * a16[2]


def _samples(params, plans):
    out = []
    for kind, n, fan, N in plans:
        with arplan.Plan(n, N, "f32", kind, fan) as p:
            f = genmodel.features(p)
        out.append((f, genmodel.predict(params, f)))
    return out


def test_fit_recovers_exact_parameters():
    true = (5e-6, 1.3e-13, 1.2e-13)
    plans = [("cps", n, None, N) for n in (2, 3, 4, 8, 16)
             for N in (1 << 10, 1 << 18, 1 << 22)]
    got = genmodel.fit(_samples(true, plans))
    assert np.allclose(got, true, rtol=1e-9, atol=0)


def test_fit_is_least_squares_in_relative_error():
    # One sample is off by +10 %; relative weighting spreads the residual
    # so that no fitted sample is off by more than the perturbation.
    true = (4e-6, 1e-13, 1e-13)
    plans = [("cps", n, None, 1 << 20) for n in (2, 4, 8, 16, 32)] + \
            [("ring", n, None, 1 << 16) for n in (4, 8)]
    s = _samples(true, plans)
    s[3] = (s[3][0], s[3][1] * 1.1)
    got = genmodel.fit(s)
    rel = [abs(genmodel.predict(got, f) - t) / t for f, t in s]
    assert max(rel) < 0.1


def test_factorizations():
    assert sorted(genmodel.factorizations(8)) == [(2, 2, 2), (2, 4), (4, 2)]
    f12 = genmodel.factorizations(12)
    assert (3, 4) in f12 and (2, 2, 3) in f12 and (12,) not in f12
    assert all(int(np.prod(f)) == 12 for f in f12)
    assert genmodel.factorizations(7) == []
    assert all(len(f) <= 2 for f in genmodel.factorizations(16, max_levels=2))


@pytest.mark.parametrize("params", [(1.0, 0.0, 0.0), (0.0, 1e-13, 1e-13),
                                    (5e-6, 1.3e-13, 1.2e-13)])
@pytest.mark.parametrize("n,N", [(8, 1 << 12), (12, 1 << 20), (32, 1 << 24)])
def test_select_is_argmin_of_prediction(params, n, N):
    t, kind, fan = genmodel.select(params, n, N)
    preds = []
    for k, f in genmodel.candidates(n):
        with arplan.Plan(n, N, "f32", k, f) as p:
            preds.append(genmodel.predict(params, genmodel.features(p)))
    assert t == min(preds)
    if params[1] == 0.0:
        # Pure round count: a two-round plan (co-located PS) wins.
        assert kind == "cps"
    if params[0] == 0.0:
        # Pure bytes: a plan with no more traffic than any candidate.
        with arplan.Plan(n, N, "f32", kind, fan) as p:
            a, d, b = genmodel.features(p)
        for k, f in genmodel.candidates(n):
            with arplan.Plan(n, N, "f32", k, f) as p:
                _, d2, b2 = genmodel.features(p)
            assert d + b <= d2 + b2


@pytest.mark.parametrize("kind,n,fan", [("ring", 8, None), ("rhd", 8, None), ("cps", 16, None),
                                        ("tree", 64, (8, 8)), ("tree", 24, (2, 3, 4))])
@pytest.mark.parametrize("N", [1 << 12, 1 << 22, 1 << 24])
def test_extended_features_split_the_paper_terms(kind, n, fan, N):
    # the extended form's byte terms add up to the paper form's, and K is
    # the sum over phases of the widest step's source count
    with arplan.Plan(n, N, "f32", kind, fan) as p:
        A, D, B = genmodel.features(p)
        A2, K, Dh, Dc, Bh, Bc = genmodel.ext_features(p)
        phases = p.phases()
    assert A2 == A and Dh + Dc == D and Bh + Bc == B
    assert K == sum(max(len(s) for _, _, s, _, _ in ph) for ph in phases)
    if n * N * 4 <= genmodel.LLC_BYTES:
        assert Dh == 0 and Bh == 0          # everything stays in the cache


def test_extended_features_cache_rule():
    # co-located PS at 1 GiB: the fold reads 16 inputs from HBM and writes
    # to HBM; the broadcast reads what the fold just wrote (64 MiB, and each
    # range 15 times) from the cache and writes 960 MiB to HBM
    with arplan.Plan(16, 1 << 24, "f32", "cps") as p:
        A, K, Dh, Dc, Bh, Bc = genmodel.ext_features(p)
    S = (1 << 24) * 4
    assert (A, K) == (2, 17)
    assert (Dh, Dc) == (17 * S, 0)
    assert Bc == 15 * S and Bh == 15 * S
    # RHD at 2 GiB: the halvings write 1 GiB, 512 MiB and 256 MiB, so the
    # second and third read from HBM; the first doubling reads the 256 MiB
    # the last halving wrote from the cache
    with arplan.Plan(8, 1 << 26, "f32", "rhd") as p:
        _, K, Dh, Dc, Bh, Bc = genmodel.ext_features(p)
    assert K == 3 * 2 + 3 * 1
    assert Dc == 0 and Bc == 256 << 20


def test_nonnegative_fit_recovers_extended_parameters():
    true = (4e-6, 3e-7, 1.6e-13, 0.7e-13, 1.3e-13, 0.6e-13)
    plans = [("cps", n, None, N) for n in (2, 3, 4, 8, 16, 24)
             for N in (1 << 10, 1 << 18, 1 << 22, 1 << 24)] + \
            [("tree", 16, (4, 4), N) for N in (1 << 18, 1 << 24)]
    s = []
    for kind, n, fan, N in plans:
        with arplan.Plan(n, N, "f32", kind, fan) as p:
            f = genmodel.ext_features(p)
        s.append((f, genmodel.predict(true, f)))
    got = genmodel.fit(s, nonneg=True)
    assert np.allclose(got, true, rtol=1e-6, atol=0)


def _reference_terms(plan, cache_bytes=genmodel.LLC_BYTES):
    """The extended form's terms computed here from the step list, to check
    the library's: per phase, the widest step's source count, and each read
    and write counted as served from the cache (whole footprint fits, or a
    range read earlier in the phase, or written by a previous phase that
    wrote at most cache_bytes) or from HBM."""
    e = plan.esize
    fits = plan.n * plan.N * e <= cache_bytes
    K = Dh = Dc = Bh = Bc = 0
    prev_written, prev_bytes = set(), 0
    phases = plan.phases()
    for ph in phases:
        K += max(len(srcs) for _, _, srcs, _, _ in ph)
        seen, written, wbytes, h, c = set(), set(), 0, 0, 0
        for op, dst, srcs, b, end in ph:
            L = (end - b) * e
            for q in srcs:
                if fits or (q, b, end) in seen or \
                        ((q, b, end) in prev_written and prev_bytes <= cache_bytes):
                    c += L
                else:
                    h += L
                seen.add((q, b, end))
            if fits:
                c += L
            else:
                h += L
            written.add((dst, b, end))
            wbytes += L
        if any(op == "reduce" for op, *_ in ph):
            Dh, Dc = Dh + h, Dc + c
        else:
            Bh, Bc = Bh + h, Bc + c
        prev_written, prev_bytes = written, wbytes
    return len(phases), K, Dh, Dc, Bh, Bc


@pytest.mark.parametrize("kind,n,fan", [("ring", 5, None), ("rhd", 6, None), ("rb", 4, None),
                                        ("cps", 9, None), ("tree", 24, (2, 3, 4))])
@pytest.mark.parametrize("N,cache", [(1000, 0), (1 << 20, 1 << 22), (1 << 22, 256 << 20)])
def test_library_terms_match_reference(kind, n, fan, N, cache):
    with arplan.Plan(n, N, "f32", kind, fan) as p:
        got = arplan.ar_genmodel_terms(p.handle, cache)
        assert tuple(int(x) for x in got) == _reference_terms(p, cache)


def test_library_select_is_argmin():
    params = (3.85e-6, 2.92e-7, 2.44e-13, 1.79e-13, 0.0, 7.68e-14)
    for n, N in ((8, 1 << 12), (12, 1 << 20), (32, 1 << 22), (7, 1000), (1, 10)):
        t, kind, fan = genmodel.select(params, n, N, feature_fn=genmodel.ext_features)
        preds = []
        for k, f in genmodel.candidates(n):
            with arplan.Plan(n, N, "f32", k, f) as p:
                preds.append((genmodel.predict(params, genmodel.ext_features(p)), k, f))
        best = min(preds, key=lambda x: x[0])     # first of equal minima
        assert (t, kind, fan) == best, (n, N)
    with pytest.raises(arplan.ArError):
        arplan.ar_genmodel_select(0, 10, "f32", params, 0)
    with pytest.raises(arplan.ArError):
        arplan.ar_genmodel_select(8, 10, "f32", params, 0, max_levels=1)


@pytest.mark.parametrize("kind,n,fan", [("ring", 5, None), ("rhd", 6, None), ("cps", 9, None),
                                        ("tree", 24, (2, 3, 4)), ("tree", 64, (8, 8))])
@pytest.mark.parametrize("N", [1000, 1 << 16, 1 << 20])
def test_tiered_terms_split_the_cached_bytes(kind, n, fan, N):
    # two tiers (the last-level cache, then the L2s): HBM bytes as with the
    # larger cache alone, tier-1 bytes what the smaller cache alone classes as
    # cached, tier-0 bytes the rest of the larger cache's cached bytes (each
    # one-cache term from the reference classification above)
    big, small = 256 << 20, 32 << 20
    with arplan.Plan(n, N, "f32", kind, fan) as p:
        t1 = arplan.ar_genmodel_terms_tiered(p.handle, [big])
        t2 = arplan.ar_genmodel_terms_tiered(p.handle, [big, small])
        rb, rs = _reference_terms(p, big), _reference_terms(p, small)
    assert tuple(int(x) for x in t1) == rb
    A, K, Dh, Dc, Dl, Bh, Bc, Bl = (int(x) for x in t2)
    assert (A, K, Dh, Bh) == (rb[0], rb[1], rb[2], rb[4])
    assert Dl == rs[3] and Dc == rb[3] - rs[3] and Bl == rs[5] and Bc == rb[5] - rs[5]
    assert min(Dc, Dl, Bc, Bl) >= 0


def test_tiered_terms_reject_bad_tiers():
    with arplan.Plan(8, 1000, "f32", "rhd") as p:
        for tiers in ([], [32 << 20, 256 << 20], [1 << 20, 1 << 20], [-1], [5, 4, 3, 2, 1]):
            with pytest.raises(arplan.ArError):
                arplan.ar_genmodel_terms_tiered(p.handle, tiers)
    with pytest.raises(arplan.ArError):
        arplan.ar_genmodel_select_tiered(8, 1000, "f32", [1.0] * 8, [1 << 20, 1 << 21])


def test_library_select_tiered_is_argmin():
    params = (2.3e-6, 5.3e-7, 2.41e-13, 1.55e-13, 1.01e-13, 0.0, 1.15e-13, 6.53e-14)
    tiers = [genmodel.LLC_BYTES, genmodel.L2_BYTES]
    for n, N in ((8, 1 << 12), (12, 1 << 20), (32, 1 << 22), (16, 1 << 18), (1, 10)):
        t, kind, fan = genmodel.select(params, n, N, feature_fn=genmodel.tiered_features)
        preds = []
        for k, f in genmodel.candidates(n):
            with arplan.Plan(n, N, "f32", k, f) as p:
                preds.append((genmodel.predict(params, genmodel.tiered_features(p, tiers)), k, f))
        best = min(preds, key=lambda x: x[0])
        assert (kind, fan) == (best[1], best[2]) and t == pytest.approx(best[0], rel=1e-12), (n, N)
    # one tier: the same choice as ar_genmodel_select
    p6 = (3.85e-6, 2.92e-7, 2.44e-13, 1.79e-13, 0.0, 7.68e-14)
    assert arplan.ar_genmodel_select_tiered(12, 1 << 20, "f32", p6, [256 << 20]) == \
        arplan.ar_genmodel_select(12, 1 << 20, "f32", p6, 256 << 20)
