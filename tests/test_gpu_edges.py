"""GPU edge cases of the cache step and the C ABI's error paths on a live
cache (state unchanged after every rejected call)."""
import ctypes

import numpy as np
import pytest

from oracle import OracleCache, attend, round_to_bf16
from paper_2606_10671_amd.synth import NumpyWanStream

from parity import check_attention, check_entries, check_state, to_np

pytestmark = pytest.mark.gpu


def make(M=3, H=2, D=128, N=96, dtype="bf16", beta=0.3, anchor=True, layers=1):
    import torch
    from paper_2606_10671_amd.fademem import Cache
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    return Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=beta, anchor=anchor, dtype=td,
                 layers=layers), OracleCache(budget=M, beta=beta, anchor=anchor, storage=dtype)


def dev(x, dtype="bf16"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda", torch.bfloat16 if dtype == "bf16" else torch.float32)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("q_tokens,cur_tokens", [(1, 5), (130, 0), (257, 1), (64, 200)])
def test_ragged_queries_and_current_chunk(dtype, q_tokens, cur_tokens):
    """Query counts off the tile size, no current chunk, a one-row chunk."""
    H, D, N = 2, 64, 80
    cache, oc = make(M=4, H=H, D=D, N=N, dtype=dtype)
    gen = NumpyWanStream(3, N, H, D)
    for t in range(6):
        k, v = gen.frame()
        cache.insert(dev(k, dtype), dev(v, dtype), t)
        cache.consolidate()
        oc.update(k, v, t)
    q = gen.queries(q_tokens)
    kc = np.concatenate([gen.frame()[0] for _ in range(3)])[:cur_tokens]
    vc = np.concatenate([gen.frame()[1] for _ in range(3)])[:cur_tokens]
    import torch
    lse = torch.empty((H, q_tokens), dtype=torch.float32, device="cuda")
    out = cache.attend(dev(q, dtype), dev(kc, dtype), dev(vc, dtype), lse=lse)
    O_ref, L_ref = attend(q, *oc.exposed_kv(), kc.reshape(cur_tokens, H, D), vc.reshape(cur_tokens, H, D))
    check_attention(to_np(out), to_np(lse), O_ref, L_ref, dtype)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_empty_memory_attends_current_chunk_only(dtype):
    H, D, N = 3, 128, 50
    cache, _ = make(M=2, H=H, D=D, N=N, dtype=dtype)
    gen = NumpyWanStream(4, N, H, D)
    q = gen.queries(70)
    kc, vc = gen.frame()
    out = cache.attend(dev(q, dtype), dev(kc, dtype), dev(vc, dtype))
    O_ref, L_ref = attend(q, [], [], kc, vc)
    check_attention(to_np(out), None, O_ref, L_ref, dtype)


@pytest.mark.parametrize("N", [1, 10, 63, 64, 65])
def test_short_entries_general_row_path(N):
    """Entries shorter than a 64-key tile (several entries per tile) use the
    kernel's general row resolution; N = 64 and 65 bracket the fast path."""
    H, D = 2, 128
    cache, oc = make(M=5, H=H, D=D, N=N)
    gen = NumpyWanStream(5, N, H, D)
    for t in range(9):
        k, v = gen.frame()
        cache.insert(dev(k), dev(v), t)
        cache.consolidate()
        oc.update(k, v, t)
    q = gen.queries(100)
    kc, vc = gen.frame()
    import torch
    lse = torch.empty((H, 100), dtype=torch.float32, device="cuda")
    out = cache.attend(dev(q), dev(kc), dev(vc), lse=lse)
    O_ref, L_ref = attend(q, *oc.exposed_kv(), kc, vc)
    check_attention(to_np(out), to_np(lse), O_ref, L_ref, "bf16")
    check_state(cache, oc)
    check_entries(cache, oc)


def test_merge_rounding_ties_and_identity():
    """Equal spans merge to the exact midpoint rounded to nearest even: two
    adjacent bf16 numbers have a midpoint that is a tie; identical blocks
    merge to themselves (anchor off, so the first merge is weighted)."""
    H, D, N = 1, 64, 64
    cache, oc = make(M=2, H=H, D=D, N=N, anchor=False, beta=0.5)
    rng = np.random.default_rng(9)
    a = round_to_bf16(rng.standard_normal((N, H, D)))
    bits = (a.view(np.uint32) >> 16).astype(np.uint32)
    b = ((bits + 1) << 16).astype(np.uint32).view(np.float32)     # next bf16 up: midpoints are ties
    c = a.copy()
    for t, blk in enumerate([a, b, c]):
        cache.insert(dev(blk), dev(blk), t)
        cache.consolidate()
        oc.update(blk, blk, t)
    assert oc.merge_log == [0]
    check_state(cache, oc)
    check_entries(cache, oc)
    k0, _ = cache.entry_kv(0, 0)
    got = to_np(k0)
    even = np.where((bits & 1) == 0, a, b)          # ties go to the even bf16 pattern
    assert np.array_equal(got.view(np.uint32), even.view(np.uint32))


def test_abi_errors_leave_state_unchanged():
    import torch
    from paper_2606_10671_amd import fademem as fm
    H, D, N, M = 1, 64, 32, 2
    cache, oc = make(M=M, H=H, D=D, N=N)
    gen = NumpyWanStream(6, N, H, D)
    frames = [gen.frame() for _ in range(4)]
    for t in range(3):
        cache.insert(dev(frames[t][0]), dev(frames[t][1]), 10 + t)
        oc.insert(frames[t][0], frames[t][1], 10 + t)
    # M+1 entries held: another insert must wait for a consolidation
    with pytest.raises(fm.FademError) as e:
        cache.insert(dev(frames[3][0]), dev(frames[3][1]), 20)
    assert e.value.code == fm.FADEMEM_ESTATE
    cache.consolidate()
    oc.consolidate()
    # positions must strictly increase
    with pytest.raises(fm.FademError) as e:
        cache.insert(dev(frames[3][0]), dev(frames[3][1]), 12)
    assert e.value.code == fm.FADEMEM_ESTATE
    # misaligned pointer, bad layer, bad scale
    L = fm.lib()
    k = dev(frames[3][0])
    bad = (ctypes.c_void_p * 1)(k.data_ptr() + 2)
    good = (ctypes.c_void_p * 1)(k.data_ptr())
    assert L.fademem_insert(ctypes.c_void_p(cache.handle), bad, good, 30, None) == fm.FADEMEM_EINVAL
    q = dev(gen.queries(8))
    out = torch.empty_like(q)
    assert L.fademem_attend(ctypes.c_void_p(cache.handle), 1, ctypes.c_void_p(q.data_ptr()), 8, None, None, 0,
                            ctypes.c_float(0), ctypes.c_void_p(out.data_ptr()), None, None) == fm.FADEMEM_EINVAL
    assert L.fademem_attend(ctypes.c_void_p(cache.handle), 0, ctypes.c_void_p(q.data_ptr()), 8, None, None, 0,
                            ctypes.c_float(-1.0), ctypes.c_void_p(out.data_ptr()), None, None) == fm.FADEMEM_EINVAL
    # consolidate within budget is a no-op
    cache.consolidate()
    check_state(cache, oc)
    check_entries(cache, oc)
    assert cache.count() == M
    # the cache still works after the rejected calls
    cache.insert(dev(frames[3][0]), dev(frames[3][1]), 21)
    cache.consolidate()
    oc.update(frames[3][0], frames[3][1], 21)
    check_state(cache, oc)
    check_entries(cache, oc)


def test_explicit_scale_and_null_lse():
    import torch
    H, D, N = 2, 128, 70
    cache, oc = make(M=3, H=H, D=D, N=N)
    gen = NumpyWanStream(7, N, H, D)
    for t in range(5):
        k, v = gen.frame()
        cache.insert(dev(k), dev(v), t)
        cache.consolidate()
        oc.update(k, v, t)
    q = gen.queries(90)
    kc, vc = gen.frame()
    out = cache.attend(dev(q), dev(kc), dev(vc), scale=0.05)
    O_ref, L_ref = attend(q, *oc.exposed_kv(), kc, vc, scale=float(np.float32(0.05)))
    check_attention(to_np(out), None, O_ref, L_ref, "bf16")


@pytest.mark.parametrize("fused", [False, True])
def test_maximum_budget(fused):
    """M = 1023, the largest budget (the schedule runs over 1024 entries in
    one block): 1100 frames of 4 tokens, state and every entry bit for bit,
    then attention over 1023 entries through the short-entry row path."""
    import torch
    from paper_2606_10671_amd.fademem import Cache
    H, D, N, M, T, F = 1, 64, 4, 1023, 1100, 4
    print(f"max budget M={M} N={N} frames={T} fused={fused}", flush=True)
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=torch.bfloat16)
    oc = OracleCache(budget=M, beta=0.3, anchor=True, storage="bf16")
    gen = NumpyWanStream(31, N, H, D)
    frames = [gen.frame() for _ in range(T)]
    kd = torch.from_numpy(np.concatenate([f[0] for f in frames])).to("cuda", torch.bfloat16)
    vd = torch.from_numpy(np.concatenate([f[1] for f in frames])).to("cuda", torch.bfloat16)
    for t0 in range(0, T, F):
        if fused:
            cache.update(kd[t0 * N:(t0 + F) * N], vd[t0 * N:(t0 + F) * N], t0)
        else:
            for t in range(t0, t0 + F):
                cache.insert(kd[t * N:(t + 1) * N], vd[t * N:(t + 1) * N], t)
                cache.consolidate()
        for t in range(t0, t0 + F):
            oc.update(frames[t][0], frames[t][1], t)
    check_state(cache, oc)
    check_entries(cache, oc)
    total, log = cache.merge_log()
    assert total == T - M and log == oc.merge_log[-len(log):]
    q = gen.queries(96)
    kc, vc = gen.frame()
    lse = torch.empty((H, 96), dtype=torch.float32, device="cuda")
    out = cache.attend(dev(q), dev(kc), dev(vc), lse=lse)
    O_ref, L_ref = attend(q, *oc.exposed_kv(), kc, vc)
    check_attention(to_np(out), to_np(lse), O_ref, L_ref, "bf16")


def test_more_layers_than_one_launch():
    """70 layers: inserts, merges and fused updates go out in launches of at
    most 64 layers; layers 0, 63, 64 and 69 are checked against the oracle."""
    import torch
    from paper_2606_10671_amd.fademem import Cache
    H, D, N, M, F, L = 1, 64, 16, 3, 2, 70
    print(f"layers={L} M={M} N={N}", flush=True)
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.5, anchor=False, dtype=torch.bfloat16,
                  layers=L)
    track = (0, 63, 64, 69)
    ocs = {l: OracleCache(budget=M, beta=0.5, anchor=False, storage="bf16") for l in track}
    gens = [NumpyWanStream(40 + l, N, H, D) for l in range(L)]
    for c in range(7):
        frames = [[g.frame() for _ in range(F)] for g in gens]
        kch = [dev(np.concatenate([f[0] for f in fr])) for fr in frames]
        vch = [dev(np.concatenate([f[1] for f in fr])) for fr in frames]
        if c % 2:
            cache.update(kch, vch, c * F)
        else:
            for f in range(F):
                cache.insert([k[f * N:(f + 1) * N] for k in kch], [v[f * N:(f + 1) * N] for v in vch], c * F + f)
                cache.consolidate()
        for l in track:
            for f in range(F):
                ocs[l].update(frames[l][f][0], frames[l][f][1], c * F + f)
        check_state(cache, ocs[0], where=c)
    for l in track:
        check_entries(cache, ocs[l], layer=l, where=l)
        q = gens[l].queries(40)
        out = cache.attend(dev(q), kch[l], vch[l], layer=l)
        K = np.concatenate([f[0] for f in frames[l]])
        V = np.concatenate([f[1] for f in frames[l]])
        O_ref, L_ref = attend(q, *ocs[l].exposed_kv(), K, V)
        check_attention(to_np(out), None, O_ref, L_ref, "bf16", where=l)
