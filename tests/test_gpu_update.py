"""GPU parity of the fused chunk update (fademem_update): a chunk's F
Algorithm S1 updates (append frame f, consolidate when over budget) in one
call, each changed K/V block written once and merged frames read straight
from the caller's chunk.

The oracle runs the same F updates one by one (Alg. S1 as written); the
schedule state, the merge log, the merge counts and every stored K/V bit
must match after every chunk.  A second GPU cache fed the same chunks
through fademem_insert + fademem_consolidate must hold the same bits too.
Cases: every consolidation operator, fp32 and bf16, anchor on and off,
beta with exact ties (1.0, 0.5), budgets from 2 (more frames per chunk than
entries) up, chunks longer than one plan (5 and 9 frames), one frame per
chunk, several layers, fills that never consolidate, and a call mixed with
the single-frame calls.
"""
import ctypes

import numpy as np
import pytest

from oracle import OracleCache
from paper_2606_10671_amd.synth import NumpyWanStream

from parity import check_attention, check_entries, check_state, oracle_attend, to_np

pytestmark = pytest.mark.gpu


def bits_equal(a, b):
    return np.array_equal(to_np(a).view(np.uint32), to_np(b).view(np.uint32))


def run(dtype="bf16", operator="sqrt_span", H=2, D=64, N=48, F=3, M=5, chunks=12, anchor=True, beta=0.3,
        layers=2, seed=11, attend_every=4):
    import torch
    from paper_2606_10671_amd.fademem import Cache
    print(f"update dtype={dtype} op={operator} H={H} D={D} N={N} F={F} M={M} chunks={chunks} anchor={anchor} "
          f"beta={beta} layers={layers}", flush=True)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    kw = dict(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=beta, anchor=anchor, dtype=td, layers=layers,
              merge_op=operator)
    fused, single = Cache(**kw), Cache(**kw)
    ocs = [OracleCache(budget=M, beta=beta, anchor=anchor, storage=dtype, operator=operator) for _ in range(layers)]
    streams = [NumpyWanStream(seed + 5 * l, N, H, D) for l in range(layers)]
    for c in range(chunks):
        frames = [[s.frame() for _ in range(F)] for s in streams]
        Ks = [np.concatenate([f[0] for f in fr]) for fr in frames]
        Vs = [np.concatenate([f[1] for f in fr]) for fr in frames]
        kd = [torch.from_numpy(np.ascontiguousarray(x)).to("cuda", td) for x in Ks]
        vd = [torch.from_numpy(np.ascontiguousarray(x)).to("cuda", td) for x in Vs]
        if c % attend_every == attend_every - 1:
            q = streams[0].queries(F * N)
            qd = torch.from_numpy(q).to("cuda", td)
            lse = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
            out = fused.attend(qd, kd[0], vd[0], layer=0, lse=lse)
            O_ref, L_ref = oracle_attend(ocs[0], q, Ks[0], Vs[0])
            check_attention(to_np(out), to_np(lse), O_ref, L_ref, dtype, where=("attend", c))
        fused.update(kd, vd, c * F)
        for f in range(F):
            single.insert([k[f * N:(f + 1) * N] for k in kd], [v[f * N:(f + 1) * N] for v in vd], c * F + f)
            single.consolidate()
            for l in range(layers):
                ocs[l].update(frames[l][f][0], frames[l][f][1], c * F + f)
        check_state(fused, ocs[0], where=c)
        assert fused.count() == len(ocs[0].entries)
        for l in range(layers):
            check_entries(fused, ocs[l], layer=l, where=(c, l))
            for i in range(len(ocs[l].entries)):
                kf, vf = fused.entry_kv(l, i)
                ks, vs = single.entry_kv(l, i)
                assert bits_equal(kf, ks) and bits_equal(vf, vs), (c, l, i)
    total, log = fused.merge_log()
    assert total == len(ocs[0].merge_log) and log == ocs[0].merge_log[-len(log):]
    assert fused.merge_counts() == single.merge_counts() == (len(ocs[0].merge_log), ocs[0].anchor_merges)
    return fused, ocs


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("operator", ["sqrt_span", "average", "select_nearest", "max"])
def test_update_operators(operator, dtype):
    run(dtype=dtype, operator=operator)


@pytest.mark.parametrize("M,F,anchor,beta", [(2, 3, True, 0.3), (2, 3, False, 1.0), (3, 5, True, 0.5),
                                             (4, 9, False, 0.3), (8, 1, True, 0.3), (21, 3, True, 0.3),
                                             (6, 4, True, 1.0)])
def test_update_budgets_and_chunk_lengths(M, F, anchor, beta):
    run(M=M, F=F, anchor=anchor, beta=beta, chunks=max(10, (3 * M) // F + 4), layers=1, H=1, D=128, N=40)


def test_update_fill_without_consolidation():
    # 2 chunks of 3 frames into a budget of 8: no merge at all, frames copied.
    _, ocs = run(M=8, F=3, chunks=2, layers=1)
    assert ocs[0].merge_log == []


def test_update_mixed_with_single_frame_calls():
    import torch
    from paper_2606_10671_amd.fademem import Cache
    H, D, N, M, F = 2, 64, 32, 4, 3
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=torch.bfloat16)
    oc = OracleCache(budget=M, beta=0.3, anchor=True, storage="bf16")
    gen = NumpyWanStream(21, N, H, D)
    t = 0
    for c in range(8):
        frames = [gen.frame() for _ in range(F)]
        if c % 2:
            k = torch.from_numpy(np.concatenate([f[0] for f in frames])).to("cuda", torch.bfloat16)
            v = torch.from_numpy(np.concatenate([f[1] for f in frames])).to("cuda", torch.bfloat16)
            cache.update(k, v, t)
        else:
            for f, (kf, vf) in enumerate(frames):
                cache.insert(torch.from_numpy(kf).to("cuda", torch.bfloat16),
                             torch.from_numpy(vf).to("cuda", torch.bfloat16), t + f)
                cache.consolidate()
        for f, (kf, vf) in enumerate(frames):
            oc.update(kf, vf, t + f)
        t += F + 2  # positions may skip
        check_state(cache, oc, where=c)
        check_entries(cache, oc, where=c)


def test_update_errors_leave_state_unchanged():
    import torch
    from paper_2606_10671_amd import fademem as fm
    from paper_2606_10671_amd.fademem import Cache
    H, D, N, M = 1, 64, 32, 3
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=torch.bfloat16)
    oc = OracleCache(budget=M, beta=0.3, anchor=True, storage="bf16")
    gen = NumpyWanStream(4, N, H, D)
    frames = [gen.frame() for _ in range(8)]
    chunk = lambda i, n: (torch.from_numpy(np.concatenate([f[0] for f in frames[i:i + n]])).to("cuda", torch.bfloat16),
                          torch.from_numpy(np.concatenate([f[1] for f in frames[i:i + n]])).to("cuda", torch.bfloat16))
    k, v = chunk(0, 3)
    cache.update(k, v, 5)
    for f in range(3):
        oc.update(frames[f][0], frames[f][1], 5 + f)
    L = fm.lib()
    k2, v2 = chunk(3, 2)
    kp = (ctypes.c_void_p * 1)(k2.data_ptr())
    vp = (ctypes.c_void_p * 1)(v2.data_ptr())
    h = ctypes.c_void_p(cache.handle)
    assert L.fademem_update(h, kp, vp, 2, 7, None) == fm.FADEMEM_ESTATE      # not above the newest (7)
    assert L.fademem_update(h, kp, vp, 0, 10, None) == fm.FADEMEM_EINVAL     # no frames
    bad = (ctypes.c_void_p * 1)(k2.data_ptr() + 4)
    assert L.fademem_update(h, bad, vp, 2, 10, None) == fm.FADEMEM_EINVAL    # misaligned
    assert L.fademem_update(h, kp, vp, 2, (1 << 40) - 1, None) == fm.FADEMEM_EINVAL  # last position out of range
    assert L.fademem_update(None, kp, vp, 2, 10, None) == fm.FADEMEM_EINVAL
    # M+1 entries held after a bare insert: the fused update must wait too
    cache.insert(torch.from_numpy(frames[3][0]).to("cuda", torch.bfloat16),
                 torch.from_numpy(frames[3][1]).to("cuda", torch.bfloat16), 9)
    assert L.fademem_update(h, kp, vp, 2, 10, None) == fm.FADEMEM_ESTATE
    cache.consolidate()
    oc.update(frames[3][0], frames[3][1], 9)
    check_state(cache, oc)
    check_entries(cache, oc)
    cache.update(k2, v2, 10)
    for f in range(2):
        oc.update(frames[3 + f][0], frames[3 + f][1], 10 + f)
    check_state(cache, oc)
    check_entries(cache, oc)


def test_update_wan_shape_thirty_layers():
    """Wan-1.3B-class shape, 30 layers in one cache, 12 chunks through the
    fused update (the memory fills after 7); head 3 of layers 0 and 29
    tracked by the oracle, bit for bit, plus attention on sampled rows."""
    import torch
    from paper_2606_10671_amd.fademem import Cache
    from paper_2606_10671_amd.synth import TorchWanStream
    from oracle import attend
    from parity import BF16_LSE_ABS, BF16_MAX_ABS, BF16_NORM_RTOL
    H, D, N, F, M, L, chunks, head = 12, 128, 1560, 3, 21, 30, 12, 3
    print(f"update wan H={H} D={D} N={N} F={F} M={M} layers={L} chunks={chunks}", flush=True)
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=torch.bfloat16,
                  layers=L)
    streams = [TorchWanStream(100 + l, N, H, D) for l in range(L)]
    ocs = {l: OracleCache(budget=M, beta=0.3, anchor=True, storage="bf16") for l in (0, L - 1)}
    for c in range(chunks):
        data = [s.chunk(F) for s in streams]
        if c == chunks - 1:
            rows = np.sort(np.random.default_rng(c).choice(F * N, size=32, replace=False))
            idx = torch.from_numpy(rows).to("cuda")
            for l, oc in ocs.items():
                q, k, v = data[l]
                lse = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
                out = cache.attend(q, k, v, layer=l, lse=lse)
                Km, Vm = oc.exposed_kv()
                O_ref, L_ref = attend(to_np(q[idx, head:head + 1]), Km, Vm, to_np(k[:, head:head + 1]),
                                      to_np(v[:, head:head + 1]))
                O = to_np(out[idx, head:head + 1]).astype(np.float64)
                err = np.abs(O - O_ref).max()
                norm = np.linalg.norm(O - O_ref) / np.linalg.norm(O_ref)
                lerr = np.abs(to_np(lse[head, idx]).astype(np.float64) - L_ref[0]).max()
                assert err <= BF16_MAX_ABS and norm <= BF16_NORM_RTOL and lerr <= BF16_LSE_ABS, (l, err, norm, lerr)
        cache.update([d[1] for d in data], [d[2] for d in data], c * F)
        for l, oc in ocs.items():
            for f in range(F):
                oc.update(to_np(data[l][1][f * N:(f + 1) * N, head:head + 1]),
                          to_np(data[l][2][f * N:(f + 1) * N, head:head + 1]), c * F + f)
        check_state(cache, ocs[0], where=c)
    for l, oc in ocs.items():
        check_entries(cache, oc, layer=l, head_slice=slice(head, head + 1))
    assert cache.merge_counts() == (len(ocs[0].merge_log), ocs[0].anchor_merges)
