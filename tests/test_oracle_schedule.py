"""Pins of the oracle's schedule and metadata (Sec. 3.1, Sec. 3.3, Alg. S1).

Every check here is independent of the oracle's own arithmetic: invariants
the paper fixes, closed forms, an exact rational schedule at beta = 1, a
60-digit schedule at other beta, and traces worked by hand.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
from mpmath import mp, mpf

from oracle import OracleCache

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def scalar_run(M, beta, anchor, positions, storage="f32"):
    """Run the oracle on scalar blocks K = V = position; return the cache and
    the list of selected indices (None when no merge was needed)."""
    c = OracleCache(budget=M, beta=beta, anchor=anchor, storage=storage)
    log = []
    for t in positions:
        x = np.array([float(t)], np.float32)
        c.insert(x, x, t)
        assert len(c.entries) <= M + 1
        log.append(c.consolidate())
        assert len(c.entries) <= M
    return c, log


CASES = [(2, 0.3, True), (3, 1.0, False), (8, 0.3, True), (8, 0.3, False), (12, 0.5, True),
         (21, 0.3, True), (21, 0.9, False), (5, 0.1, True), (16, 0.7, True)]


@pytest.mark.parametrize("M,beta,anchor", CASES)
def test_budget_span_sum_and_order(M, beta, anchor):
    """P1-P3: |M_t| <= M (Sec. 3.1), spans sum to the number of inserted
    blocks and the covered ranges tile the history (Sec. 3.3: s counts the
    units an entry summarises), order is preserved (only adjacent pairs
    merge, Sec. 3.3)."""
    rng = np.random.default_rng(M * 1000 + int(beta * 10))
    positions = np.cumsum(rng.integers(1, 4, size=150)).tolist()  # strictly increasing, with skips
    c, _ = scalar_run(M, beta, anchor, positions)
    inserted = len(positions)
    assert sum(e.span for e in c.entries) == inserted
    firsts = [e.first for e in c.entries]
    assert firsts == sorted(set(firsts))
    assert firsts[0] == positions[0]
    bounds = firsts + [positions[-1] + 1]
    pos = np.array(positions)
    for i, e in enumerate(c.entries):
        covered = pos[(pos >= bounds[i]) & (pos < bounds[i + 1])]
        assert e.span == len(covered)
        if e.anchor:
            assert e.pos_sum == e.first * e.span
        else:
            assert e.pos_sum == int(covered.sum())       # s*mu = sum of covered positions
    mus = [Fraction(e.pos_sum, e.span) for e in c.entries]
    assert all(a < b for a, b in zip(mus, mus[1:]))


@pytest.mark.parametrize("M,beta,anchor", CASES)
def test_newest_entry_protected(M, beta, anchor):
    """P5: after every update the last entry is the just-inserted block,
    untouched (Sec. 3.3 boundary handling, Alg. S1 eligible pairs)."""
    c = OracleCache(budget=M, beta=beta, anchor=anchor)
    rng = np.random.default_rng(7)
    for t in range(60):
        K = rng.standard_normal((3, 2)).astype(np.float32)
        V = rng.standard_normal((3, 2)).astype(np.float32)
        c.insert(K, V, t)
        c.consolidate()
        last = c.entries[-1]
        assert (last.first, last.pos_sum, last.span) == (t, t, 1)
        assert np.array_equal(last.K.view(np.uint32), K.view(np.uint32))
        assert np.array_equal(last.V.view(np.uint32), V.view(np.uint32))


@pytest.mark.parametrize("M,beta", [(3, 1.0), (8, 0.3), (21, 0.3), (12, 0.9)])
def test_anchor_kept_bitwise(M, beta):
    """P6: with the anchor on, entry 0 keeps the first block's K, V bitwise
    and its position forever (Alg. S1 anchor branch, supplementary S1)."""
    rng = np.random.default_rng(3)
    K0 = rng.standard_normal((4, 3)).astype(np.float32)
    V0 = rng.standard_normal((4, 3)).astype(np.float32)
    c = OracleCache(budget=M, beta=beta, anchor=True)
    c.insert(K0, V0, 5)
    for t in range(6, 200):
        c.update(rng.standard_normal((4, 3)).astype(np.float32),
                 rng.standard_normal((4, 3)).astype(np.float32), t)
        a = c.entries[0]
        assert a.anchor and a.first == 5 and a.pos_sum == 5 * a.span
        assert np.array_equal(a.K, K0) and np.array_equal(a.V, V0)
    assert c.anchor_merges > 0
    assert not any(e.anchor for e in c.entries[1:])


@pytest.mark.parametrize("M", [2, 3, 8, 12, 21])
@pytest.mark.parametrize("beta", [0.1, 0.3, 0.5, 0.9])
def test_first_merge_closed_form(M, beta):
    """P7: no merge while fewer than M+1 blocks are held; with 0-indexed
    consecutive positions the first merge (at t = M) picks the oldest pair,
    because u(d) = d**beta is strictly concave for beta < 1, so gaps between
    consecutive integers shrink with distance.  Anchor on: the anchor
    absorbs block 1 and keeps K = block 0.  Anchor off: the two blocks are
    averaged with w = 1/2, i.e. the exact midpoint."""
    for anchor in (True, False):
        c, log = scalar_run(M, beta, anchor, range(M + 1))
        assert log[:M] == [None] * M
        assert log[M] == 0
        e0 = c.entries[0]
        assert e0.span == 2
        if anchor:
            assert e0.K[0] == 0.0 and e0.pos_sum == 0
        else:
            assert e0.K[0] == 0.5 and e0.pos_sum == 1


def exact_schedule_beta1(M, anchor, T):
    """Independent exact schedule at beta = 1: u(d) = d, so the gap of pair
    (i, i+1) is mu_{i+1} - mu_i, held as exact fractions; ties to the lowest
    index.  The anchor's mu stays at its first position."""
    mus, spans, anc = [], [], []
    js = []
    for t in range(T):
        mus.append(Fraction(t)); spans.append(1); anc.append(anchor and t == 0)
        if len(mus) <= M:
            js.append(None)
            continue
        g = [mus[i + 1] - mus[i] for i in range(len(mus) - 2)]
        j = g.index(min(g))
        s = spans[j] + spans[j + 1]
        mu = mus[j] if anc[j] else (spans[j] * mus[j] + spans[j + 1] * mus[j + 1]) / s
        mus[j:j + 2] = [mu]; spans[j:j + 2] = [s]; anc[j:j + 2] = [anc[j]]
        js.append(j)
    return js, spans


@pytest.mark.parametrize("M,anchor,T", [(3, False, 200), (8, True, 400), (8, False, 400),
                                        (21, True, 3000), (21, False, 1500)])
def test_beta_one_matches_exact_rationals(M, anchor, T):
    """P8: at beta = 1 the fp64 schedule (with its tie tolerance) equals an
    exact rational schedule at every step, exact ties included."""
    js_exact, spans_exact = exact_schedule_beta1(M, anchor, T)
    c, log = scalar_run(M, 1.0, anchor, range(T))
    assert log == js_exact
    assert [e.span for e in c.entries] == spans_exact


def hp_schedule(M, beta, anchor, T, digits=60, tie_rtol=1e-9):
    """Independent 60-digit schedule with exact rational distances.  Near
    ties within tie_rtol (relative) go to the lowest index, the reading the
    oracle uses.  Also returns the smallest relative margin between the best
    and second-best gap among non-tied steps."""
    mp.dps = digits
    b = mpf(beta)
    firsts, psums, spans, anc = [], [], [], []
    js, margin = [], None
    for t in range(T):
        firsts.append(t); psums.append(t); spans.append(1); anc.append(anchor and t == 0)
        if len(spans) <= M:
            js.append(None)
            continue
        d = [mpf(t * s - p) / s for s, p in zip(spans[:-1], psums[:-1])]
        u = [x ** b for x in d]
        g = [abs(u[i + 1] - u[i]) for i in range(len(spans) - 2)]
        gm = min(g)
        j = next(i for i, gi in enumerate(g) if gi - gm <= tie_rtol * gm)
        others = sorted(float((gi - gm) / gm) for gi in g if gi - gm > tie_rtol * gm)
        if others:
            margin = others[0] if margin is None else min(margin, others[0])
        s = spans[j] + spans[j + 1]
        p = firsts[j] * s if anc[j] else psums[j] + psums[j + 1]
        firsts[j:j + 2] = [firsts[j]]; psums[j:j + 2] = [p]; spans[j:j + 2] = [s]; anc[j:j + 2] = [anc[j]]
        js.append(j)
    return js, margin


@pytest.mark.parametrize("beta", [0.1, 0.3, 0.5, 0.7, 0.9])
@pytest.mark.parametrize("M,anchor,T", [(8, True, 300), (21, True, 700), (21, False, 400)])
def test_fp64_schedule_matches_high_precision(beta, M, anchor, T):
    """P9: the fp64 schedule equals a 60-digit schedule at every step, and
    non-tied decisions have a margin far above fp64 rounding."""
    js_hp, margin = hp_schedule(M, beta, anchor, T)
    _, log = scalar_run(M, beta, anchor, range(T))
    assert log == js_hp
    assert margin is None or margin > 1e-7


def test_hand_traces():
    """Traces worked by hand from Sec. 3.3 / Alg. S1 (tests/golden)."""
    with open(os.path.join(GOLDEN, "hand_traces.json")) as f:
        traces = json.load(f)["traces"]
    mp.dps = 40
    for tr in traces:
        c, log = scalar_run(tr["budget"], tr["beta"], tr["anchor"], range(tr["inserts"]))
        assert [j for j in log if j is not None] == tr["j"], tr["name"]
        st = c.state()
        assert st["first"] == tr["first"] and st["span"] == tr["span"] and st["pos_sum"] == tr["pos_sum"]
        for e, v in zip(c.entries, tr["values"]):
            exact = mpf(v)
            got = float(e.K[0])
            ulp = float(np.spacing(np.float32(abs(float(exact)))))
            assert abs(mpf(got) - exact) <= mpf(ulp) * 0.5 + mpf(2) ** -60, (tr["name"], got, v)
            assert e.K[0] == e.V[0]


def spans_non_increasing_with_recency(c):
    """Spans of non-anchor entries, oldest first, must not increase."""
    s = [e.span for e in c.entries if not e.anchor]
    return all(a >= b for a, b in zip(s, s[1:]))


@pytest.mark.parametrize("M,T,anchor", [(8, 40, True), (8, 40, False), (21, 360, True), (21, 360, False)])
def test_spans_grow_with_distance_on_workload_runs(M, T, anchor):
    """Sec. 3.3: the memory becomes a hierarchy whose older entries cover
    longer spans.  On the tiny (M=8, 40 steps) and Wan-class (M=21, 120
    chunks of 3 frames) runs at beta = 0.3 every step has spans that do not
    increase from older to newer (non-anchor entries)."""
    c = OracleCache(budget=M, beta=0.3, anchor=anchor)
    z = np.zeros(1, np.float32)
    for t in range(T):
        c.update(z, z, t)
        assert spans_non_increasing_with_recency(c), t


def test_span_order_is_not_a_strict_invariant():
    """The paper states the hierarchy qualitatively (Sec. 3.3); Alg. S1 does
    not enforce it.  Over long runs an adjacent newer entry can briefly
    cover more units than its older neighbour (bounded here by 2x).  This
    test keeps anyone from 'fixing' the oracle to force the order."""
    c = OracleCache(budget=8, beta=0.3, anchor=True)
    z = np.zeros(1, np.float32)
    violated = False
    for t in range(400):
        c.update(z, z, t)
        s = [e.span for e in c.entries if not e.anchor]
        if not all(a >= b for a, b in zip(s, s[1:])):
            violated = True
        assert all(b <= 2 * a for a, b in zip(s, s[1:]))
    assert violated


def test_merge_log_and_counters_m21():
    """Counters: every update past the budget merges exactly once."""
    c = OracleCache(budget=21, beta=0.3, anchor=True)
    z = np.zeros(1, np.float32)
    for t in range(360):
        c.update(z, z, t)
    assert len(c.merge_log) == 360 - 21
    assert c.anchor_merges + c.weighted_merges == 360 - 21
    assert sum(e.span for e in c.entries) == 360


def test_insert_rejects_bad_calls():
    c = OracleCache(budget=2, beta=0.3)
    z = np.zeros(1, np.float32)
    c.insert(z, z, 0)
    with pytest.raises(ValueError):
        c.insert(z, z, 0)            # not strictly increasing
    c.insert(z, z, 1); c.insert(z, z, 2)
    with pytest.raises(ValueError):
        c.insert(z, z, 3)            # budget+1 entries pending a consolidation
    with pytest.raises(ValueError):
        OracleCache(budget=1)
    with pytest.raises(ValueError):
        OracleCache(budget=4, beta=0.0)
    with pytest.raises(ValueError):
        OracleCache(budget=4, beta=1.5)
