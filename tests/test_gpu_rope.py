"""GPU parity of attention with temporal RoPE handling (Sec. 3.3 "Boundary
and positional handling"): memory keys stored without their temporal phase,
entry i exposed at temporal index i, the current chunk at n + f.

The caller's side (queries and current keys rotated to n + f) is done here
with the oracle's rotation; the library rotates the memory.  Attention is
compared with the oracle (memory keys rotated to their entry index and
rounded to the storage type, then fp64 attention) within the bf16 / fp32
bars, and the stored (phase-free) entries bit for bit.  Parity unpinned as
to the paper's index mapping, which the paper does not state.
"""
import numpy as np
import pytest

from oracle import OracleCache, attend, exposed_kv_rope, rope_rotate
from paper_2606_10671_amd.synth import NumpyWanStream

from parity import check_attention, check_entries, check_state, to_np

pytestmark = pytest.mark.gpu


def run(dtype, D, pairs, H=2, N=56, F=2, M=4, chunks=8, theta=10000.0, seed=9, fused=True, q_scale=1.0):
    import torch
    from paper_2606_10671_amd.fademem import Cache
    print(f"rope dtype={dtype} D={D} pairs={pairs} H={H} N={N} F={F} M={M} chunks={chunks}", flush=True)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=td,
                  rope_pairs=pairs, rope_theta=theta)
    oc = OracleCache(budget=M, beta=0.3, anchor=True, storage=dtype)
    gen = NumpyWanStream(seed, N, H, D)
    for c in range(chunks):
        frames = [gen.frame() for _ in range(F)]
        K = np.concatenate([f[0] for f in frames])
        V = np.concatenate([f[1] for f in frames])
        Q = gen.queries(F * N) * q_scale
        n = len(oc.entries)
        # caller side: queries and current keys at temporal indices n + f
        Qr = np.concatenate([rope_rotate(Q[f * N:(f + 1) * N], n + f, pairs, theta, dtype) for f in range(F)])
        Kr = np.concatenate([rope_rotate(K[f * N:(f + 1) * N], n + f, pairs, theta, dtype) for f in range(F)])
        qd, kd, vd, krd = (torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda", td)
                           for x in (Qr, K, V, Kr))
        lse = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
        out = cache.attend(qd, krd, vd, lse=lse)
        Km, Vm = exposed_kv_rope(oc, pairs, theta)
        O_ref, L_ref = attend(Qr, Km, Vm, Kr, V)
        check_attention(to_np(out), to_np(lse), O_ref, L_ref, dtype, where=(c, pairs))
        # memory update with the phase-free keys
        if fused:
            cache.update(kd, vd, c * F)
        else:
            for f in range(F):
                cache.insert(kd[f * N:(f + 1) * N], vd[f * N:(f + 1) * N], c * F + f)
                cache.consolidate()
        for f in range(F):
            oc.update(frames[f][0], frames[f][1], c * F + f)
        check_state(cache, oc, where=c)
        check_entries(cache, oc, where=c)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("D,pairs", [(64, 1), (64, 32), (128, 22), (128, 64)])
def test_rope_attention(dtype, D, pairs):
    run(dtype, D, pairs)


def test_rope_peaked_softmax_single_frame_updates():
    # Scaled queries make the weights peaked, so a key rotated to the wrong
    # index would move the output by much more than the bars.
    run("bf16", 128, 22, q_scale=6.0, fused=False, chunks=6)


def test_rope_wan_shape():
    """Wan-1.3B-class shape with Wan's temporal axis (22 of 64 pairs)."""
    import torch
    from paper_2606_10671_amd.fademem import Cache
    from paper_2606_10671_amd.synth import TorchWanStream
    from parity import BF16_LSE_ABS, BF16_MAX_ABS, BF16_NORM_RTOL
    H, D, N, F, M, P, chunks, head = 12, 128, 1560, 3, 21, 22, 9, 4
    print(f"rope wan H={H} N={N} F={F} M={M} P={P} chunks={chunks}", flush=True)
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=torch.bfloat16,
                  rope_pairs=P)
    oc = OracleCache(budget=M, beta=0.3, anchor=True, storage="bf16")
    stream = TorchWanStream(77, N, H, D)
    for c in range(chunks):
        q, k, v = stream.chunk(F)
        if c == chunks - 1:
            n = len(oc.entries)
            qn, kn = to_np(q[:, head:head + 1]), to_np(k[:, head:head + 1])
            rows = np.sort(np.random.default_rng(c).choice(F * N, size=32, replace=False))
            # rotate this head's queries and current keys on the host, others left as they are
            qr = np.concatenate([rope_rotate(qn[f * N:(f + 1) * N], n + f, P, 10000.0, "bf16") for f in range(F)])
            kr = np.concatenate([rope_rotate(kn[f * N:(f + 1) * N], n + f, P, 10000.0, "bf16") for f in range(F)])
            qd, kd = q.clone(), k.clone()
            qd[:, head:head + 1] = torch.from_numpy(qr).to("cuda", torch.bfloat16)
            kd[:, head:head + 1] = torch.from_numpy(kr).to("cuda", torch.bfloat16)
            lse = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
            out = cache.attend(qd, kd, v, lse=lse)
            Km, Vm = exposed_kv_rope(oc, P, 10000.0)
            O_ref, L_ref = attend(qr[rows], Km, Vm, kr, to_np(v[:, head:head + 1]))
            O = to_np(out[torch.from_numpy(rows).to("cuda"), head:head + 1]).astype(np.float64)
            err = np.abs(O - O_ref).max()
            norm = np.linalg.norm(O - O_ref) / np.linalg.norm(O_ref)
            lerr = np.abs(to_np(lse[head, torch.from_numpy(rows).to("cuda")]).astype(np.float64) - L_ref[0]).max()
            print(f"max-abs {err:.3e} normwise {norm:.3e} lse {lerr:.3e}", flush=True)
            assert err <= BF16_MAX_ABS and norm <= BF16_NORM_RTOL and lerr <= BF16_LSE_ABS
        cache.update(k, v, c * F)
        for f in range(F):
            oc.update(to_np(k[f * N:(f + 1) * N, head:head + 1]), to_np(v[f * N:(f + 1) * N, head:head + 1]),
                      c * F + f)
    check_state(cache, oc)
    check_entries(cache, oc, head_slice=slice(head, head + 1))


def test_rope_attend_between_insert_and_consolidate():
    """With M + 1 entries held (after an insert, before its consolidation)
    the re-indexed view exposes all of them, entry M at index M."""
    import torch
    from paper_2606_10671_amd.fademem import Cache
    H, D, N, M, P, steps = 2, 128, 72, 4, 22, 12
    print(f"rope insert-then-attend H={H} N={N} M={M} P={P} steps={steps}", flush=True)
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=torch.bfloat16,
                  rope_pairs=P)
    oc = OracleCache(budget=M, beta=0.3, anchor=True, storage="bf16")
    gen = NumpyWanStream(5, N, H, D)
    seen_full = False
    for t in range(steps):
        k, v = gen.frame()
        kd, vd = (torch.from_numpy(np.ascontiguousarray(x)).to("cuda", torch.bfloat16) for x in (k, v))
        cache.insert(kd, vd, t)
        oc.insert(k, v, t)
        n = len(oc.entries)
        seen_full = seen_full or n == M + 1
        q = gen.queries(N)
        qr = rope_rotate(q, n, P, 10000.0, "bf16")       # the caller's chunk at index n
        kc, vc = gen.frame()
        kcr = rope_rotate(kc, n, P, 10000.0, "bf16")
        qd, kcd, vcd = (torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda", torch.bfloat16)
                        for x in (qr, kcr, vc))
        lse = torch.empty((H, N), dtype=torch.float32, device="cuda")
        out = cache.attend(qd, kcd, vcd, lse=lse)
        Km, Vm = exposed_kv_rope(oc, P, 10000.0)
        O_ref, L_ref = attend(qr, Km, Vm, kcr, vc)
        check_attention(to_np(out), to_np(lse), O_ref, L_ref, "bf16", where=("held", n))
        cache.consolidate()
        oc.consolidate()
        cache.verify()
        check_state(cache, oc, where=t)
    assert seen_full


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_rope_views_per_layer_across_denoising_steps(dtype):
    """Several layers, each attended several times per chunk (one call per
    denoising step) before the update: every call must see its own layer's
    memory re-indexed, whichever layer was attended last."""
    import torch
    from paper_2606_10671_amd.fademem import Cache
    H, D, N, F, M, P, L, chunks, steps = 2, 64, 40, 2, 4, 11, 3, 7, 3
    print(f"rope layers={L} steps={steps} dtype={dtype}", flush=True)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=td, layers=L,
                  rope_pairs=P)
    ocs = [OracleCache(budget=M, beta=0.3, anchor=True, storage=dtype) for _ in range(L)]
    gens = [NumpyWanStream(40 + l, N, H, D) for l in range(L)]
    for c in range(chunks):
        frames = [[g.frame() for _ in range(F)] for g in gens]
        Ks = [np.concatenate([f[0] for f in fr]) for fr in frames]
        Vs = [np.concatenate([f[1] for f in fr]) for fr in frames]
        n = len(ocs[0].entries)
        for s in range(steps):
            for l in (range(L) if s % 2 == 0 else reversed(range(L))):
                q = gens[l].queries(F * N)
                qr = np.concatenate([rope_rotate(q[f * N:(f + 1) * N], n + f, P, 10000.0, dtype) for f in range(F)])
                kr = np.concatenate([rope_rotate(Ks[l][f * N:(f + 1) * N], n + f, P, 10000.0, dtype)
                                     for f in range(F)])
                qd, krd, vd = (torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to("cuda", td)
                               for x in (qr, kr, Vs[l]))
                lse = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
                out = cache.attend(qd, krd, vd, layer=l, lse=lse)
                Km, Vm = exposed_kv_rope(ocs[l], P, 10000.0)
                O_ref, L_ref = attend(qr, Km, Vm, kr, Vs[l])
                check_attention(to_np(out), to_np(lse), O_ref, L_ref, dtype, where=(c, s, l))
        kd = [torch.from_numpy(np.ascontiguousarray(x)).to("cuda", td) for x in Ks]
        vd = [torch.from_numpy(np.ascontiguousarray(x)).to("cuda", td) for x in Vs]
        cache.update(kd, vd, c * F)
        for l in range(L):
            for f in range(F):
                ocs[l].update(frames[l][f][0], frames[l][f][1], c * F + f)
        check_state(cache, ocs[0], where=c)
    cache.verify()
