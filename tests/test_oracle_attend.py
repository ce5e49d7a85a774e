"""Pins of the oracle's attention (Sec. 3.1: the chunk's queries attend over
[memory || current chunk]; textbook softmax attention)."""
import math

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import OracleCache, attend, chunk_step


def brute(Q, K, V, scale):
    """Pure-Python loops with math.exp: softmax(q.k * scale) weighted sum."""
    Lq, H, D = Q.shape
    Lk = K.shape[0]
    O = np.zeros((Lq, H, D))
    for h in range(H):
        for i in range(Lq):
            s = [sum(float(Q[i, h, d]) * float(K[j, h, d]) for d in range(D)) * scale for j in range(Lk)]
            w = [math.exp(x) for x in s]
            tot = sum(w)
            for d in range(D):
                O[i, h, d] = sum(w[j] * float(V[j, h, d]) for j in range(Lk)) / tot
    return O


def test_matches_brute_force_on_tiny_inputs():
    rng = np.random.default_rng(0)
    H, D, N = 2, 4, 3
    Q = rng.standard_normal((5, H, D))
    Km = [rng.standard_normal((N, H, D)) for _ in range(2)]
    Vm = [rng.standard_normal((N, H, D)) for _ in range(2)]
    Kc, Vc = rng.standard_normal((4, H, D)), rng.standard_normal((4, H, D))
    O, LSE = attend(Q, Km, Vm, Kc, Vc)
    Kall = np.concatenate(Km + [Kc]); Vall = np.concatenate(Vm + [Vc])
    ref = brute(Q, Kall, Vall, 1 / math.sqrt(D))
    assert np.allclose(O, ref, rtol=1e-12, atol=1e-12)
    for h in range(H):
        S = Q[:, h] @ Kall[:, h].T / math.sqrt(D)
        assert np.allclose(LSE[h], logsumexp(S, axis=1), rtol=1e-13, atol=1e-13)


def test_single_key_returns_its_value():
    rng = np.random.default_rng(1)
    Q = rng.standard_normal((7, 3, 8))
    Kc, Vc = rng.standard_normal((1, 3, 8)), rng.standard_normal((1, 3, 8))
    O, _ = attend(Q, [], [], Kc, Vc)
    assert np.allclose(O, np.broadcast_to(Vc, O.shape), rtol=0, atol=1e-15)


def test_zero_query_gives_the_mean_value():
    rng = np.random.default_rng(2)
    Km = [rng.standard_normal((6, 2, 4))]
    Vm = [rng.standard_normal((6, 2, 4))]
    Kc, Vc = rng.standard_normal((3, 2, 4)), rng.standard_normal((3, 2, 4))
    O, LSE = attend(np.zeros((2, 2, 4)), Km, Vm, Kc, Vc)
    mean = np.concatenate([Vm[0], Vc]).mean(axis=0)
    assert np.allclose(O, np.broadcast_to(mean, O.shape), atol=1e-14)
    assert np.allclose(LSE, math.log(9.0), atol=1e-14)


def test_key_permutation_invariance_and_scale():
    rng = np.random.default_rng(3)
    Q = rng.standard_normal((4, 1, 16))
    K, V = rng.standard_normal((20, 1, 16)), rng.standard_normal((20, 1, 16))
    perm = rng.permutation(20)
    O1, L1 = attend(Q, [K[:10]], [V[:10]], K[10:], V[10:], scale=0.7)
    O2, L2 = attend(Q, [], [], K[perm], V[perm], scale=0.7)
    assert np.allclose(O1, O2, atol=1e-13) and np.allclose(L1, L2, atol=1e-13)
    O3, _ = attend(Q, [], [], K, V)                       # default 1/sqrt(D)
    O4, _ = attend(Q, [], [], K, V, scale=0.25)
    assert np.allclose(O3, O4, atol=1e-15)


def test_query_blocking_is_invisible():
    rng = np.random.default_rng(4)
    Q = rng.standard_normal((37, 2, 8))
    K, V = rng.standard_normal((11, 2, 8)), rng.standard_normal((11, 2, 8))
    O1, L1 = attend(Q, [], [], K, V, q_block=5)
    O2, L2 = attend(Q, [], [], K, V, q_block=1024)
    assert np.array_equal(O1, O2) and np.array_equal(L1, L2)


def test_chunk_step_attends_before_inserting():
    """The chunk's own frames are passed as 'current' keys; the memory
    update happens after attention (Sec. 4.1), one update per frame."""
    rng = np.random.default_rng(5)
    c = OracleCache(budget=2, beta=0.3)
    H, D, N, F = 1, 4, 2, 3
    seen = []

    def spy(Q, Km, Vm, Kc, Vc):
        seen.append((len(Km), Kc.shape[0]))
        return attend(Q, Km, Vm, Kc, Vc)
    for ch in range(3):
        K = rng.standard_normal((F * N, H, D)).astype(np.float32)
        V = rng.standard_normal((F * N, H, D)).astype(np.float32)
        _, _, merges = chunk_step(c, rng.standard_normal((F * N, H, D)), K, V, F, ch * F, attend_fn=spy)
        assert len(merges) == F
        assert np.array_equal(c.entries[-1].K, K[(F - 1) * N:])
    assert seen == [(0, 6), (2, 6), (2, 6)]
