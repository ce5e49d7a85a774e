"""Hour-scale run at the Wan-1.3B-class shape: 30 layers in one cache,
4800 chunks of 3 frames (14 400 frames, about an hour of video at 16 fps
with a 4x temporal VAE), budget 21, beta 0.3, anchor on, bf16.

Every frame is drawn from one seeded AR(1) stream with N + 29 token rows;
layer l inserts rows [l, l + N).  Merges are elementwise, so a single oracle
run over the tall frames (one tracked head) fixes every layer's merged K/V:
entry i of layer l must equal rows [l, l + N) of the oracle's entry i, bit
for bit.  The schedule state (int64 positions, spans, pos_sums) is checked
against the oracle along the run and at the end, the merge log at the end,
and attention of the last chunk on sampled query rows of layers 0 and 29.

The run is made three ways: one fademem_insert + fademem_consolidate per
frame, one fused fademem_update per chunk (the benchmark's path: its plan
kernel's merge log wraps past its 4096-entry ring and its counters grow to
14 379 consolidations), and the zero-copy staged update, whose host replay
of the slot table is checked against the device along the run.
"""
import numpy as np
import pytest

from oracle import OracleCache, attend
from parity import BF16_LSE_ABS, BF16_MAX_ABS, BF16_NORM_RTOL, check_state, to_np

pytestmark = pytest.mark.gpu

H, D, N, F, M, L, CHUNKS = 12, 128, 1560, 3, 21, 30, 4800
HEAD = 5


@pytest.mark.parametrize("update", ["single", "fused", "staged"])
def test_hour_scale_thirty_layers(update):
    import torch
    from paper_2606_10671_amd.fademem import Cache
    from paper_2606_10671_amd.synth import TorchWanStream
    print(f"hour-scale H={H} D={D} N={N} F={F} M={M} layers={L} chunks={CHUNKS} update={update}", flush=True)
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=torch.bfloat16,
                  layers=L, stage_frames=F if update == "staged" else 0)
    blk = N * H * D * 2
    # Peak cache bytes: M+1 slots per layer of K and V (M+F when staging),
    # plus metadata and the attention scratch.
    slots = M + (F if update == "staged" else 1)
    assert slots * L * 2 * blk <= cache.pool_bytes <= slots * L * 2 * blk + 128 * 2**20
    print(f"pool bytes {cache.pool_bytes}", flush=True)
    stream = TorchWanStream(7, N + L - 1, H, D)
    oc = OracleCache(budget=M, beta=0.3, anchor=True, storage="bf16")
    for c in range(CHUNKS):
        frames = [stream.frame() for _ in range(F)]
        if c == CHUNKS - 1:
            q = torch.randn((F * N, H, D), device="cuda").to(torch.bfloat16)
            rows = np.sort(np.random.default_rng(c).choice(F * N, size=48, replace=False))
            idx = torch.from_numpy(rows).to("cuda")
            for layer in (0, L - 1):
                kc = torch.cat([k[layer:layer + N] for k, _ in frames]).contiguous()
                vc = torch.cat([v[layer:layer + N] for _, v in frames]).contiguous()
                out = torch.empty_like(q)
                lse = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
                cache.attend(q, kc, vc, layer=layer, out=out, lse=lse)
                km = [e.K[layer:layer + N] for e in oc.entries]
                vm = [e.V[layer:layer + N] for e in oc.entries]
                O_ref, L_ref = attend(to_np(q[idx, HEAD:HEAD + 1]), km, vm, to_np(kc[:, HEAD:HEAD + 1]),
                                      to_np(vc[:, HEAD:HEAD + 1]))
                O = to_np(out[idx, HEAD:HEAD + 1]).astype(np.float64)
                err = np.abs(O - O_ref).max()
                norm = np.linalg.norm(O - O_ref) / np.linalg.norm(O_ref)
                lerr = np.abs(to_np(lse[HEAD, idx]).astype(np.float64) - L_ref[0]).max()
                print(f"last chunk layer {layer}: max-abs {err:.3e} normwise {norm:.3e} lse {lerr:.3e}", flush=True)
                assert err <= BF16_MAX_ABS and norm <= BF16_NORM_RTOL and lerr <= BF16_LSE_ABS, (layer, err, norm,
                                                                                                lerr)
        if update == "single":
            for f, (k, v) in enumerate(frames):
                cache.insert([k[layer:layer + N] for layer in range(L)], [v[layer:layer + N] for layer in range(L)],
                             c * F + f)
                cache.consolidate()
        elif update == "fused":
            cache.update([torch.cat([k[layer:layer + N] for k, _ in frames]) for layer in range(L)],
                         [torch.cat([v[layer:layer + N] for _, v in frames]) for layer in range(L)], c * F)
        else:
            staged = cache.stage(F)
            for layer in range(L):
                for f, (k, v) in enumerate(frames):
                    staged[layer][f][0].copy_(k[layer:layer + N])
                    staged[layer][f][1].copy_(v[layer:layer + N])
            cache.update_staged(F, c * F)
        for f, (k, v) in enumerate(frames):
            oc.update(to_np(k[:, HEAD:HEAD + 1]), to_np(v[:, HEAD:HEAD + 1]), c * F + f)
        if c % 400 == 0 or c == CHUNKS - 1:
            check_state(cache, oc, where=c)
            if update == "staged":
                cache.verify()
            print(f"chunk {c}: state matches ({len(oc.merge_log)} consolidations, "
                  f"{oc.anchor_merges} anchor merges)", flush=True)
    st = cache.state()
    assert st["newest"] == CHUNKS * F - 1 and sum(st["span"]) == CHUNKS * F
    total, log = cache.merge_log()
    assert total == len(oc.merge_log) == CHUNKS * F - M
    assert log == oc.merge_log[-len(log):]
    assert cache.merge_counts() == (len(oc.merge_log), oc.anchor_merges)
    for i, e in enumerate(oc.entries):
        for layer in range(L):
            kk, vv = cache.entry_kv(layer, i)
            kr = e.K[layer:layer + N].view(np.uint32)
            vr = e.V[layer:layer + N].view(np.uint32)
            assert np.array_equal(to_np(kk[:, HEAD:HEAD + 1]).view(np.uint32), kr), (layer, i, "K")
            assert np.array_equal(to_np(vv[:, HEAD:HEAD + 1]).view(np.uint32), vr), (layer, i, "V")
    print(f"final spans {st['span']}", flush=True)
