"""GPU parity of the zero-copy update (Alg. S1 "Append"; Sec. 4.1 and
supplementary Sec. S4: one entry per latent frame, the memory updated once
the chunk is generated).

The caller writes a chunk's frames straight into the staging slots that
fademem_stage hands out, attends over [memory || staged frames]
(fademem_attend_staged) and then runs the chunk's F Alg. S1 updates
(fademem_update_staged).  The oracle runs the same updates one by one;
schedule state, merge log and every stored K/V bit must match after every
chunk, as must a second cache fed the same chunks through fademem_update
(the caller's buffers, kept frames copied).  Attention is compared with the
oracle within the bars, and the library's host replay of the slot table is
checked against the device (fademem_verify) after every chunk.
"""
import numpy as np
import pytest

from oracle import OracleCache, attend, exposed_kv_rope, rope_rotate
from paper_2606_10671_amd.synth import NumpyWanStream

from parity import check_attention, check_entries, check_state, oracle_attend, to_np

pytestmark = pytest.mark.gpu


def bits_equal(a, b):
    return np.array_equal(to_np(a).view(np.uint32), to_np(b).view(np.uint32))


def run(dtype="bf16", H=2, D=128, N=96, F=3, M=5, chunks=14, operator="sqrt_span", anchor=True, beta=0.3,
        layers=2, rope_pairs=0, seed=21, q_scale=1.0):
    import torch
    from paper_2606_10671_amd.fademem import Cache
    print(f"staged dtype={dtype} H={H} D={D} N={N} F={F} M={M} chunks={chunks} op={operator} anchor={anchor} "
          f"beta={beta} layers={layers} rope={rope_pairs}", flush=True)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    kw = dict(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=beta, anchor=anchor, dtype=td, layers=layers,
              merge_op=operator, rope_pairs=rope_pairs)
    staged, ref = Cache(**kw, stage_frames=F), Cache(**kw)
    ocs = [OracleCache(budget=M, beta=beta, anchor=anchor, storage=dtype, operator=operator) for _ in range(layers)]
    streams = [NumpyWanStream(seed + 7 * l, N, H, D) for l in range(layers)]
    for c in range(chunks):
        frames = [[s.frame() for _ in range(F)] for s in streams]
        Ks = [np.concatenate([f[0] for f in fr]) for fr in frames]
        Vs = [np.concatenate([f[1] for f in fr]) for fr in frames]
        kd = [torch.from_numpy(np.ascontiguousarray(x)).to("cuda", td) for x in Ks]
        vd = [torch.from_numpy(np.ascontiguousarray(x)).to("cuda", td) for x in Vs]
        slots = staged.stage(F)
        for l in range(layers):
            for f in range(F):
                slots[l][f][0].copy_(kd[l][f * N:(f + 1) * N])
                slots[l][f][1].copy_(vd[l][f * N:(f + 1) * N])
        # the final pass over the chunk: attention over [memory || staged frames]
        n = len(ocs[0].entries)
        q = streams[0].queries(F * N) * np.float32(q_scale)
        for l in range(layers):
            if rope_pairs:
                qr = np.concatenate([rope_rotate(q[f * N:(f + 1) * N], n + f, rope_pairs, 10000.0, dtype)
                                     for f in range(F)])
                kr = np.concatenate([rope_rotate(Ks[l][f * N:(f + 1) * N], n + f, rope_pairs, 10000.0, dtype)
                                     for f in range(F)])
                Km, Vm = exposed_kv_rope(ocs[l], rope_pairs, 10000.0)
                O_ref, L_ref = attend(qr, Km, Vm, kr, Vs[l])
            else:
                qr = q
                O_ref, L_ref = oracle_attend(ocs[l], q, Ks[l], Vs[l])
            qd = torch.from_numpy(np.ascontiguousarray(qr, dtype=np.float32)).to("cuda", td)
            lse = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
            out = staged.attend_staged(qd, F, layer=l, lse=lse)
            check_attention(to_np(out), to_np(lse), O_ref, L_ref, dtype, where=("attend_staged", c, l))
        staged.update_staged(F, c * F)
        ref.update(kd, vd, c * F)
        for l in range(layers):
            for f in range(F):
                ocs[l].update(frames[l][f][0], frames[l][f][1], c * F + f)
        staged.verify()
        check_state(staged, ocs[0], where=c)
        assert staged.state() == ref.state()
        for l in range(layers):
            check_entries(staged, ocs[l], layer=l, where=(c, l))
            for i in range(len(ocs[l].entries)):
                ks, vs = staged.entry_kv(l, i)
                kr_, vr_ = ref.entry_kv(l, i)
                assert bits_equal(ks, kr_) and bits_equal(vs, vr_), (c, l, i)
    total, log = staged.merge_log()
    assert total == len(ocs[0].merge_log) and log == ocs[0].merge_log[-len(log):]
    assert staged.merge_counts() == ref.merge_counts() == (len(ocs[0].merge_log), ocs[0].anchor_merges)
    return staged


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("operator", ["sqrt_span", "select_nearest", "max"])
def test_staged_update_operators(dtype, operator):
    run(dtype=dtype, operator=operator, D=64 if dtype == "f32" else 128)


@pytest.mark.parametrize("F,M", [(1, 2), (2, 2), (4, 3), (3, 21)])
def test_staged_frames_and_budgets(F, M):
    """Budgets from 2 (more staged frames than entries) up; one to four frames."""
    run(F=F, M=M, chunks=12 if M < 10 else 10, N=40 if M > 10 else 96)


@pytest.mark.parametrize("beta,anchor", [(1.0, True), (0.5, False)])
def test_staged_with_exact_ties(beta, anchor):
    """Schedules with exact ties: the host replay must take the same (lowest) pair."""
    run(beta=beta, anchor=anchor, chunks=20, N=48)


def test_staged_with_rope():
    """Temporal RoPE handling with staged frames: they are exposed at n + f
    (the library rotates them, as the caller wrote them phase-free)."""
    run(rope_pairs=22, chunks=10)


def test_staged_peaked_softmax():
    """Peaked weights: a staged frame read from the wrong slot would move the
    output far beyond the bars."""
    run(q_scale=8.0, chunks=8, layers=1)


def test_stage_rejects_bad_requests():
    import torch
    from paper_2606_10671_amd.fademem import Cache, FademError, FADEMEM_EINVAL, FADEMEM_ESTATE
    cache = Cache(budget=3, heads=2, head_dim=64, tokens_per_block=64, dtype=torch.bfloat16, stage_frames=2)
    plain = Cache(budget=3, heads=2, head_dim=64, tokens_per_block=64, dtype=torch.bfloat16)
    with pytest.raises(FademError) as e:
        cache.stage(3)                    # more frames than configured
    assert e.value.code == FADEMEM_EINVAL
    with pytest.raises(FademError) as e:
        plain.stage(1)                    # staging off
    assert e.value.code == FADEMEM_EINVAL
    k = torch.zeros((64, 2, 64), dtype=torch.bfloat16, device="cuda")
    for t in range(4):                    # M + 1 entries held: stage must wait for the consolidation
        cache.insert(k, k, t)
    with pytest.raises(FademError) as e:
        cache.stage(1)
    assert e.value.code == FADEMEM_ESTATE
    cache.consolidate()
    cache.stage(2)
    with pytest.raises(FademError) as e:
        cache.update_staged(2, 3)         # position not above the newest
    assert e.value.code == FADEMEM_ESTATE
    cache.verify()
