"""Pins of the oracle's temporal RoPE handling (Sec. 3.3 "Boundary and
positional handling").

The rotation is pinned to mathematics the oracle does not use: pairs as
complex numbers multiplied by exp(i * angle), composition of rotations,
norm preservation, the identity at index 0, and the relative-position
property that makes re-indexing possible at all (attention depends only on
index differences, so shifting every index by the same amount changes
nothing).  Which index each retained entry gets is a reading the paper does
not state: parity unpinned as to the paper's mapping.
"""
import numpy as np
import pytest

from oracle import OracleCache, attend, exposed_kv_rope, round_to_bf16, rope_angles, rope_rotate


def rng_x(seed, shape):
    return np.random.default_rng(seed).standard_normal(shape)


@pytest.mark.parametrize("pairs,theta", [(1, 10000.0), (22, 10000.0), (32, 500.0), (64, 1e6)])
def test_rotation_is_complex_multiplication(pairs, theta):
    D = 128 if pairs > 32 else 64
    X = rng_x(pairs, (5, 3, D))
    idx = 37.0
    Y = rope_rotate(X, idx, pairs, theta)
    k = np.arange(pairs)
    ang = idx * theta ** (-k / pairs)
    z = (X[..., 0:2 * pairs:2] + 1j * X[..., 1:2 * pairs:2]) * np.exp(1j * ang)
    np.testing.assert_allclose(Y[..., 0:2 * pairs:2], z.real, rtol=0, atol=1e-12)
    np.testing.assert_allclose(Y[..., 1:2 * pairs:2], z.imag, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(Y[..., 2 * pairs:], X[..., 2 * pairs:])  # other dims untouched


def test_composition_identity_and_norm():
    X = rng_x(1, (7, 2, 128))
    a = rope_rotate(rope_rotate(X, 11, 22, 10000.0), 30, 22, 10000.0)
    b = rope_rotate(X, 41, 22, 10000.0)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(rope_rotate(X, 0, 22, 10000.0), X)       # index 0: angle 0 exactly
    np.testing.assert_array_equal(rope_rotate(X, 99, 0, 10000.0), X)       # no pairs: identity
    n0 = X[..., 0:44:2] ** 2 + X[..., 1:44:2] ** 2
    n1 = b[..., 0:44:2] ** 2 + b[..., 1:44:2] ** 2
    np.testing.assert_allclose(n0, n1, rtol=1e-12)
    # the first pair turns by exactly the index (frequency theta^0 = 1)
    np.testing.assert_allclose(rope_angles(41, 22, 10000.0)[0], 41.0)


def test_storage_rounding_of_rotated_keys():
    X = round_to_bf16(rng_x(2, (4, 1, 64)))
    Y = rope_rotate(X, 5, 8, 10000.0, storage="bf16")
    np.testing.assert_array_equal(Y, round_to_bf16(rope_rotate(X, 5, 8, 10000.0)))


def test_attention_depends_only_on_index_differences():
    """Rotating every key and query by the same extra index leaves attention
    unchanged: shifting the re-indexed range does not matter."""
    H, D, N, P, theta = 2, 64, 16, 16, 10000.0
    oc = OracleCache(budget=4, beta=0.3, anchor=True, storage="f32")
    rng = np.random.default_rng(3)
    for t in range(7):
        oc.update(rng.standard_normal((N, H, D)).astype(np.float32), rng.standard_normal((N, H, D)).astype(np.float32), t)
    n = len(oc.entries)
    Q = rng.standard_normal((2 * N, H, D))
    Kc = rng.standard_normal((2 * N, H, D))
    Vc = rng.standard_normal((2 * N, H, D))

    def run(shift):
        Km = [rope_rotate(e.K, i + shift, P, theta) for i, e in enumerate(oc.entries)]
        Vm = [e.V for e in oc.entries]
        Qr = np.concatenate([rope_rotate(Q[f * N:(f + 1) * N], n + f + shift, P, theta) for f in range(2)])
        Kr = np.concatenate([rope_rotate(Kc[f * N:(f + 1) * N], n + f + shift, P, theta) for f in range(2)])
        return attend(Qr, Km, Vm, Kr, Vc)

    O0, L0 = run(0)
    O1, L1 = run(1234)
    np.testing.assert_allclose(O1, O0, rtol=0, atol=1e-10)
    np.testing.assert_allclose(L1, L0, rtol=0, atol=1e-10)
    # and the rotation matters: without it the result differs
    O2, _ = attend(Q, [e.K for e in oc.entries], [e.V for e in oc.entries], Kc, Vc)
    assert np.abs(O2 - O0).max() > 1e-3


def test_exposed_memory_uses_entry_order():
    oc = OracleCache(budget=3, beta=0.3, anchor=True, storage="bf16")
    rng = np.random.default_rng(5)
    for t in range(6):
        k = round_to_bf16(rng.standard_normal((4, 1, 64)))
        oc.update(k, k, t)
    Km, Vm = exposed_kv_rope(oc, 8, 10000.0)
    for i, e in enumerate(oc.entries):
        np.testing.assert_array_equal(Km[i], rope_rotate(e.K, i, 8, 10000.0, "bf16"))
        assert Vm[i] is e.V
