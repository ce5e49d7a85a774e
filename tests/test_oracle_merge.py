"""Pins of the oracle's consolidation operator and storage rounding
(Sec. 3.3 "Consolidation operator", Alg. S1; BF16 storage, Sec. 4.1)."""
from fractions import Fraction

import numpy as np
import pytest
import torch
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import Entry, OracleCache, bf16_bits, bf16_from_bits, round_to_bf16


def merge(storage, sa, sb, Ka, Kb):
    c = OracleCache(budget=4, beta=0.3, storage=storage)
    a = Entry(0, 0, sa, False, Ka, Ka.copy())
    b = Entry(sa, sa, sb, False, Kb, Kb.copy())
    K, V = c.merge_values(a, b)
    assert np.array_equal(K.view(np.uint32), V.view(np.uint32))
    return K


# -- bf16 rounding -----------------------------------------------------------

def test_bf16_rounding_matches_torch_on_fp32_inputs():
    """For fp32 inputs, round-to-nearest-even to bfloat16 is what torch's
    CPU conversion does: compare over every exponent, ties and subnormals."""
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 2**32, size=200_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    ties = ((rng.integers(0, 2**16, size=5000).astype(np.uint32) << 16) | 0x8000).view(np.float32)
    ties = ties[np.isfinite(ties)]
    x = np.concatenate([x, ties, np.float32([0.0, -0.0, 1.0, 3.3895314e38, -3.3895314e38, 1e-45])])
    ours = round_to_bf16(x.astype(np.float64))
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_bf16_rounding_fp64_inputs_brute_force():
    """For fp64 inputs, the result is the nearest bfloat16 number, found by
    brute force over the sorted table of all finite bfloat16 values; ties go
    to the even pattern."""
    table_bits = np.arange(0, 2**16, dtype=np.uint32).astype(np.uint16)
    vals = bf16_from_bits(table_bits)
    ok = np.isfinite(vals)
    vals, table_bits = vals[ok], table_bits[ok]
    order = np.argsort(vals.astype(np.float64), kind="stable")
    vals, table_bits = vals[order].astype(np.float64), table_bits[order]
    keep = np.concatenate([[True], np.diff(vals) > 0])    # drop -0 duplicate of +0
    vals, table_bits = vals[keep], table_bits[keep]
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-40, 38, size=20000),
                        (vals[1:-1] + vals[2:]) / 2])      # exact midpoints (ties)
    x = x[np.abs(x) < vals[-1]]
    ours = round_to_bf16(x).astype(np.float64)
    hi = np.searchsorted(vals, x, side="left")
    lo = np.clip(hi - 1, 0, len(vals) - 1)
    hi = np.clip(hi, 0, len(vals) - 1)
    dlo, dhi = np.abs(x - vals[lo]), np.abs(vals[hi] - x)
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (table_bits[hi] % 2 == 0) & (table_bits[lo] % 2 == 1))
    expect = np.where(pick_hi, vals[hi], vals[lo])
    assert np.array_equal(ours, expect)


def test_bf16_bit_helpers_round_trip():
    b = np.arange(0, 2**16, dtype=np.uint32).astype(np.uint16)
    assert np.array_equal(bf16_bits(bf16_from_bits(b)), b)


# -- consolidation operator -----------------------------------------------------

@pytest.mark.parametrize("storage", ["f32", "bf16"])
@settings(max_examples=60, deadline=None)
@given(sa=st.integers(1, 10000), sb=st.integers(1, 10000), seed=st.integers(0, 2**31))
def test_merging_identical_blocks_is_identity(storage, sa, sb, seed):
    """P4: merging a block with an identical block returns it bitwise."""
    x = np.random.default_rng(seed).standard_normal(257) * 3
    x = (round_to_bf16(x) if storage == "bf16" else x.astype(np.float32))
    K = merge(storage, sa, sb, x, x.copy())
    assert np.array_equal(K.view(np.uint32), x.view(np.uint32))


@pytest.mark.parametrize("storage", ["f32", "bf16"])
def test_equal_spans_give_the_nearest_midpoint(storage):
    """P11: s_j = s_{j+1} gives w = 1/2, so the result is the storage
    number nearest to the exact midpoint (checked with exact fractions)."""
    rng = np.random.default_rng(2)
    a = rng.standard_normal(500) * 7
    b = rng.standard_normal(500) * 7
    if storage == "bf16":
        a, b = round_to_bf16(a), round_to_bf16(b)
    else:
        a, b = a.astype(np.float32), b.astype(np.float32)
    r = merge(storage, 5, 5, a, b)
    for x, y, z in zip(a, b, r):
        mid = (Fraction(float(x)) + Fraction(float(y))) / 2
        err = abs(Fraction(float(z)) - mid)
        # neighbours of z in the storage format
        if storage == "bf16":
            bz = int(bf16_bits(np.float32([z]))[0])
            nb = [float(bf16_from_bits(np.uint16([(bz + d) & 0xFFFF]))[0]) for d in (-1, 1)]
        else:
            nb = [float(np.nextafter(z, np.float32(-np.inf))), float(np.nextafter(z, np.float32(np.inf)))]
        for n in nb:
            if np.isfinite(n):
                assert err <= abs(Fraction(n) - mid)


def test_sqrt_span_weights_orientation():
    """w_j = sqrt(s_j)/(sqrt(s_j)+sqrt(s_{j+1})): spans (1, 4) give weights
    (1/3, 2/3), so merging 0 and 3 gives 2; spans (4, 1) give 1; spans
    (9, 16) on 0 and 7 give 4."""
    z = np.zeros(3, np.float32)
    for storage in ("f32", "bf16"):
        assert np.all(merge(storage, 1, 4, z, z + 3) == 2.0)
        assert np.all(merge(storage, 4, 1, z, z + 3) == 1.0)
        assert np.all(merge(storage, 9, 16, z, z + 7) == 4.0)


@pytest.mark.parametrize("storage", ["f32", "bf16"])
@settings(max_examples=60, deadline=None)
@given(sa=st.integers(1, 5000), sb=st.integers(1, 5000), seed=st.integers(0, 2**31))
def test_merge_is_a_convex_combination(storage, sa, sb, seed):
    """Merged values lie in [min, max] of the pair, and are within half a
    storage ulp (plus fp64 slack) of the exact sqrt-span weighted mean."""
    rng = np.random.default_rng(seed)
    a, b = rng.standard_normal(64) * 4, rng.standard_normal(64) * 4
    if storage == "bf16":
        a, b = round_to_bf16(a), round_to_bf16(b)
    else:
        a, b = a.astype(np.float32), b.astype(np.float32)
    r = merge(storage, sa, sb, a, b)
    assert np.all(r >= np.minimum(a, b)) and np.all(r <= np.maximum(a, b))
    ra, rb = np.sqrt(np.longdouble(sa)), np.sqrt(np.longdouble(sb))
    wa, wb = ra / (ra + rb), rb / (ra + rb)
    exact = wa * a.astype(np.longdouble) + wb * b.astype(np.longdouble)
    # Half an ulp of the stored result (one rounding), plus the error of the
    # fp64 evaluation it rounds: a few fp64 ulps of the summands' magnitude,
    # which dominates only when the summands cancel.
    if storage == "bf16":
        ulp = np.spacing(np.abs(r)) * 2.0**16
    else:
        ulp = np.spacing(np.abs(r))
    eval_err = 2.0**-50 * (wa * np.abs(a) + wb * np.abs(b))
    assert np.all(np.abs(r.astype(np.longdouble) - exact) <= 0.5 * ulp.astype(np.longdouble) + eval_err)


def test_anchor_pair_keeps_anchor_bits_and_drops_neighbour():
    """Alg. S1 anchor branch: spans add, K, V and position of the anchor are
    kept, the neighbour's K, V are discarded."""
    c = OracleCache(budget=2, beta=0.5, anchor=True, storage="bf16")
    rng = np.random.default_rng(4)
    blocks = [round_to_bf16(rng.standard_normal((5, 2))) for _ in range(3)]
    vals = [round_to_bf16(b.astype(np.float64) + 1) for b in blocks]
    for t, (blk, val) in enumerate(zip(blocks, vals)):
        c.insert(blk, val, 10 + t)
    j = c.consolidate()
    assert j == 0
    a = c.entries[0]
    assert (a.first, a.span, a.pos_sum) == (10, 2, 20)
    assert np.array_equal(a.K, blocks[0]) and np.array_equal(a.V, vals[0])
    assert np.array_equal(c.entries[1].K, blocks[2])


# -- Table 4 operators (Sec. 4.3 "Memory consolidation operator") -------------

def merge_op(operator, storage, sa, sb, Ka, Kb, Va=None, Vb=None):
    c = OracleCache(budget=4, beta=0.3, storage=storage, operator=operator)
    a = Entry(0, 0, sa, False, Ka, Ka.copy() if Va is None else Va)
    b = Entry(sa, sa, sb, False, Kb, Kb.copy() if Vb is None else Vb)
    return c.merge_values(a, b)


def test_unknown_operator_is_rejected():
    with pytest.raises(ValueError):
        OracleCache(budget=4, operator="median")


@pytest.mark.parametrize("storage", ["f32", "bf16"])
def test_average_ignores_spans_and_gives_the_nearest_midpoint(storage):
    """Unweighted average: spans (1, 4) on (0, 3) give 1.5 (the sqrt-span
    default gives 2), and in general the storage number nearest the exact
    midpoint (exact fractions; ties to the even pattern)."""
    z = np.zeros(3, np.float32)
    K, _ = merge_op("average", storage, 1, 4, z, z + 3)
    assert np.all(K == 1.5)
    rng = np.random.default_rng(12)
    a, b = rng.standard_normal(400) * 5, rng.standard_normal(400) * 5
    a, b = (round_to_bf16(a), round_to_bf16(b)) if storage == "bf16" else (a.astype(np.float32), b.astype(np.float32))
    r, _ = merge_op("average", storage, 7, 100, a, b)
    for x, y, z_ in zip(a, b, r):
        mid = (Fraction(float(x)) + Fraction(float(y))) / 2
        if storage == "bf16":
            bz = int(bf16_bits(np.float32([z_]))[0])
            nb = [float(bf16_from_bits(np.uint16([(bz + d) & 0xFFFF]))[0]) for d in (-1, 1)]
        else:
            nb = [float(np.nextafter(z_, np.float32(-np.inf))), float(np.nextafter(z_, np.float32(np.inf)))]
        err = abs(Fraction(float(z_)) - mid)
        assert all(err <= abs(Fraction(n) - mid) for n in nb if np.isfinite(n))


def test_select_nearest_keeps_the_newer_bits():
    rng = np.random.default_rng(13)
    Ka, Kb = round_to_bf16(rng.standard_normal((4, 3))), round_to_bf16(rng.standard_normal((4, 3)))
    Va, Vb = round_to_bf16(rng.standard_normal((4, 3))), round_to_bf16(rng.standard_normal((4, 3)))
    K, V = merge_op("select_nearest", "bf16", 3, 9, Ka, Kb, Va, Vb)
    assert np.array_equal(K.view(np.uint32), Kb.view(np.uint32))
    assert np.array_equal(V.view(np.uint32), Vb.view(np.uint32))


def test_max_pooling_elementwise_and_signed_zero():
    """Elementwise maximum (brute force per element); equal values keep the
    older entry's bits, so max(-0, +0) is -0 when -0 is older."""
    rng = np.random.default_rng(14)
    Ka = round_to_bf16(rng.standard_normal(300))
    Kb = round_to_bf16(rng.standard_normal(300))
    Ka[:3] = [-0.0, 0.0, 1.0]
    Kb[:3] = [0.0, -0.0, 1.0]
    K, _ = merge_op("max", "bf16", 1, 1, Ka, Kb)
    for i in range(300):
        want = Kb[i] if float(Kb[i]) > float(Ka[i]) else Ka[i]
        assert np.float32(K[i]).view(np.uint32) == np.float32(want).view(np.uint32), i
    assert np.signbit(K[0]) and not np.signbit(K[1])


@pytest.mark.parametrize("operator", ["average", "select_nearest", "max"])
def test_operator_changes_values_not_the_schedule(operator):
    """The schedule depends only on positions (Sec. 3.3): every operator makes
    the same decisions and keeps the same metadata as the default, and the
    anchor still keeps its own K, V bits."""
    rng = np.random.default_rng(15)
    ref = OracleCache(budget=5, beta=0.3, anchor=True, storage="bf16")
    alt = OracleCache(budget=5, beta=0.3, anchor=True, storage="bf16", operator=operator)
    blocks = [round_to_bf16(rng.standard_normal((3, 2))) for _ in range(30)]
    for t, blk in enumerate(blocks):
        ref.update(blk, blk, t)
        alt.update(blk, blk, t)
    assert ref.merge_log == alt.merge_log and ref.state() == alt.state()
    assert np.array_equal(alt.entries[0].K, blocks[0])
