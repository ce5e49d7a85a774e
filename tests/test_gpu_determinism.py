"""Deterministic replay: the same seeded inputs, run twice through two
caches, give the same bits (attention outputs, metadata, every stored K/V
bit), also when one of them runs in serialize mode (FADEMEM_SERIALIZE,
each call waits for its own work).  No kernel of the path uses atomics or an
order that depends on timing."""
import numpy as np
import pytest

from paper_2606_10671_amd.synth import NumpyWanStream

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype_name,H,D,N,F,M", [("bf16", 4, 128, 160, 3, 6), ("f32", 2, 64, 64, 2, 8)])
def test_replay_is_bit_identical(dtype_name, H, D, N, F, M, monkeypatch):
    import torch
    from paper_2606_10671_amd.fademem import Cache
    dtype = torch.bfloat16 if dtype_name == "bf16" else torch.float32
    print(f"determinism {dtype_name} H={H} D={D} N={N} F={F} M={M}", flush=True)
    kw = dict(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=True, dtype=dtype)
    a = Cache(**kw)
    monkeypatch.setenv("FADEMEM_SERIALIZE", "1")
    b = Cache(**kw)
    monkeypatch.delenv("FADEMEM_SERIALIZE")
    gen = NumpyWanStream(3, N, H, D)
    bits = (lambda t: t.view(torch.uint8)) if dtype == torch.bfloat16 else (lambda t: t.view(torch.int32))
    for c in range(10):
        fr = [gen.frame() for _ in range(F)]
        q = torch.from_numpy(gen.queries(F * N)).cuda().to(dtype)
        k = torch.from_numpy(np.concatenate([f[0] for f in fr])).cuda().to(dtype)
        v = torch.from_numpy(np.concatenate([f[1] for f in fr])).cuda().to(dtype)
        la = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
        lb = torch.empty_like(la)
        oa, ob = a.attend(q, k, v, lse=la), b.attend(q, k, v, lse=lb)
        assert torch.equal(bits(oa), bits(ob)) and torch.equal(la.view(torch.int32), lb.view(torch.int32))
        a.update(k, v, c * F)
        b.update(k, v, c * F)
        sa, sb = a.state(), b.state()
        assert sa == sb
        for i in range(sa["count"]):
            for x, y in zip(a.entry_kv(0, i), b.entry_kv(0, i)):
                assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))
    assert a.merge_log() == b.merge_log()
