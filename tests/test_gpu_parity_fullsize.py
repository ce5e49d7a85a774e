"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark times (one cache, attend per layer, then F inserts+consolidates).

The oracle cannot hold a full-size run, so it follows whole heads: merges
are elementwise and attention is per head, so the library's result for a
head equals the oracle run on that head's slice alone.  It checks, bit for
bit, the schedule state after every chunk and the tracked heads' merged K/V,
and attention on sampled query rows of the tracked heads (fp64 over the
full memory) within the bf16 bars.
"""
import numpy as np
import pytest

from oracle import OracleCache, attend
from parity import BF16_LSE_ABS, BF16_MAX_ABS, BF16_NORM_RTOL, check_state, to_np

pytestmark = pytest.mark.gpu


def run_fullsize(H, D, N, F, M, chunks, layers=1, heads=(0,), check_layers=(0,), attn_chunks=(), rows=64,
                 seed=0, update="single", attend_layers=None):
    import torch
    from paper_2606_10671_amd.fademem import Cache
    from paper_2606_10671_amd.synth import TorchWanStream
    print(f"fullsize H={H} D={D} N={N} F={F} M={M} chunks={chunks} layers={layers} heads={heads} update={update}",
          flush=True)
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=torch.bfloat16,
                  layers=layers)
    streams = [TorchWanStream(seed + 1000 * l, N, H, D) for l in range(layers)]
    ocs = {(l, h): OracleCache(budget=M, beta=0.3, anchor=True, storage="bf16") for l in check_layers for h in heads}
    out = torch.empty((F * N, H, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
    rng = np.random.default_rng(seed)
    worst = [0.0, 0.0, 0.0]
    for c in range(chunks):
        data = [streams[l].chunk(F) for l in range(layers)]
        for l in range(layers) if attend_layers is None else attend_layers:
            q, k, v = data[l]
            cache.attend(q, k, v, layer=l, out=out, lse=lse)
            if c in attn_chunks and l in check_layers:
                sel = np.sort(rng.choice(F * N, size=rows, replace=False))
                idx = torch.from_numpy(sel).to("cuda")
                for h in heads:
                    qh = to_np(q[idx, h:h + 1])
                    Km, Vm = ocs[(l, h)].exposed_kv()
                    O_ref, L_ref = attend(qh, Km, Vm, to_np(k[:, h:h + 1]), to_np(v[:, h:h + 1]))
                    O = to_np(out[idx, h:h + 1]).astype(np.float64)
                    L = to_np(lse[h, idx]).astype(np.float64)
                    err = np.abs(O - O_ref).max()
                    norm = np.linalg.norm(O - O_ref) / np.linalg.norm(O_ref)
                    lerr = np.abs(L - L_ref[0]).max()
                    worst = [max(worst[0], err), max(worst[1], norm), max(worst[2], lerr)]
                    assert err <= BF16_MAX_ABS and norm <= BF16_NORM_RTOL and lerr <= BF16_LSE_ABS, (c, l, h, err,
                                                                                                   norm, lerr)
        if update == "fused":
            cache.update([data[l][1] for l in range(layers)], [data[l][2] for l in range(layers)], c * F)
        for f in range(F):
            ks = [data[l][1][f * N:(f + 1) * N] for l in range(layers)]
            vs = [data[l][2][f * N:(f + 1) * N] for l in range(layers)]
            if update == "single":
                cache.insert(ks, vs, c * F + f)
                cache.consolidate()
            for (l, h), oc in ocs.items():
                oc.update(to_np(ks[l][:, h:h + 1]), to_np(vs[l][:, h:h + 1]), c * F + f)
        check_state(cache, next(iter(ocs.values())), where=c)
    for (l, h), oc in ocs.items():
        for i, e in enumerate(oc.entries):
            kk, vv = cache.entry_kv(l, i)
            assert np.array_equal(to_np(kk[:, h:h + 1]).view(np.uint32), e.K.view(np.uint32)), (l, h, i)
            assert np.array_equal(to_np(vv[:, h:h + 1]).view(np.uint32), e.V.view(np.uint32)), (l, h, i)
    total, log = cache.merge_log()
    oc0 = next(iter(ocs.values()))
    assert total == len(oc0.merge_log) and log == oc0.merge_log[-len(log):]
    assert cache.merge_counts() == (len(oc0.merge_log), oc0.anchor_merges)
    print(f"worst max-abs {worst[0]:.3e} normwise {worst[1]:.3e} lse {worst[2]:.3e}", flush=True)
    return cache, oc0


def test_wan13b_single_layer_full_run():
    """Wan-1.3B-class layer: 12 heads x 128, 1560 tokens per frame, 3-frame
    chunks, budget 21, 120 chunks (the benchmark's workload)."""
    _, oc = run_fullsize(H=12, D=128, N=1560, F=3, M=21, chunks=120, heads=(0, 7),
                         attn_chunks=(0, 6, 7, 8, 60, 119))
    assert [e.span for e in oc.entries] == [22, 64, 32, 32, 32, 32, 32, 16, 16, 16, 16, 16, 8, 8, 4, 4, 4, 2, 2, 1, 1]


def test_wan13b_thirty_layers_one_cache():
    """All 30 layers in one cache: one schedule, one merge launch for every
    layer; layers 0 and 29 tracked."""
    run_fullsize(H=12, D=128, N=1560, F=3, M=21, chunks=12, layers=30, heads=(5,), check_layers=(0, 29),
                 attn_chunks=(11,), rows=32)


def test_14b_class_layer():
    """14B-class layer at 720p: 40 heads x 128, 3600 tokens per frame
    (10 800 queries, 86 400 keys at steady state)."""
    run_fullsize(H=40, D=128, N=3600, F=3, M=21, chunks=9, heads=(0, 39), attn_chunks=(8,), rows=32)


def test_14b_class_forty_layers_fused():
    """The 14B-class configuration as benchmarked: 40 layers in one cache
    (64.9 GB of K/V slots), 40 heads x 128, 3600 tokens per frame, fused
    chunk updates.  Layers 0 and 39 are tracked bit for bit (one head
    each) and attended on sampled rows at the last chunk, which sees the
    full memory (86 400 keys)."""
    run_fullsize(H=40, D=128, N=3600, F=3, M=21, chunks=9, layers=40, heads=(11,), check_layers=(0, 39),
                 attn_chunks=(8,), rows=32, update="fused", attend_layers=(0, 39))

