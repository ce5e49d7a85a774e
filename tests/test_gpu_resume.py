"""Checkpoint / resume: a cache restored from a snapshot of another
(fademem_get_state + each entry's K, V) continues exactly as the original:
for every later chunk the attention output, the metadata and every stored
K/V bit are equal to the uninterrupted cache's.  Also the errors of
fademem_set_state (host-side validation, before anything is enqueued)."""
import ctypes

import numpy as np
import pytest

from paper_2606_10671_amd.synth import NumpyWanStream

pytestmark = pytest.mark.gpu


def _cache(dtype, **kw):
    from paper_2606_10671_amd.fademem import Cache
    return Cache(dtype=dtype, **kw)


def _same_entries(a, b):
    import torch
    sa, sb = a.state(), b.state()
    assert sa == sb
    for l in range(a.cfg.layers):
        for i in range(sa["count"]):
            for x, y in zip(a.entry_kv(l, i), b.entry_kv(l, i)):
                assert torch.equal(x.view(torch.uint8), y.view(torch.uint8))


@pytest.mark.parametrize("dtype_name,H,D,N,F,M,layers,op,anchor", [
    ("bf16", 2, 128, 96, 2, 5, 1, "sqrt_span", True),
    ("bf16", 3, 64, 72, 3, 4, 2, "max", False),
    ("f32", 2, 64, 64, 1, 8, 1, "average", True),
])
def test_resume_continues_exactly(dtype_name, H, D, N, F, M, layers, op, anchor):
    import torch
    dtype = torch.bfloat16 if dtype_name == "bf16" else torch.float32
    print(f"resume {dtype_name} H={H} D={D} N={N} F={F} M={M} layers={layers} op={op}", flush=True)
    kw = dict(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=anchor, layers=layers,
              merge_op=op)
    a = _cache(dtype, **kw)
    gens = [NumpyWanStream(7 + l, N, H, D) for l in range(layers)]

    def chunk():
        fr = [[g.frame() for _ in range(F)] for g in gens]
        q = torch.from_numpy(gens[0].queries(F * N)).cuda().to(dtype)
        ks = [torch.from_numpy(np.concatenate([f[0] for f in fl])).cuda().to(dtype) for fl in fr]
        vs = [torch.from_numpy(np.concatenate([f[1] for f in fl])).cuda().to(dtype) for fl in fr]
        return q, ks, vs

    pos = 0
    for _ in range(6):
        q, ks, vs = chunk()
        a.update(ks, vs, pos)
        pos += F
    snap = a.snapshot()
    b = _cache(dtype, **kw)
    b.restore(snap)
    _same_entries(a, b)
    for _ in range(6):
        q, ks, vs = chunk()
        for l in range(layers):
            oa = a.attend(q, ks[l], vs[l], layer=l)
            ob = b.attend(q, ks[l], vs[l], layer=l)
            assert torch.equal(oa.view(torch.uint8) if dtype == torch.bfloat16 else oa.view(torch.int32),
                               ob.view(torch.uint8) if dtype == torch.bfloat16 else ob.view(torch.int32))
        a.update(ks, vs, pos)
        b.update(ks, vs, pos)
        pos += F
        _same_entries(a, b)
    assert b.merge_counts()[0] > 0
    # positions must keep increasing after the restore
    from paper_2606_10671_amd import fademem as fm
    with pytest.raises(fm.FademError):
        b.update(ks, vs, pos - 1)


def test_set_state_errors():
    import torch
    from paper_2606_10671_amd import fademem as fm
    kw = dict(budget=4, heads=2, head_dim=64, tokens_per_block=64, beta=0.3, anchor=True)
    a = _cache(torch.float32, **kw)
    blk = [torch.zeros((64, 2, 64), dtype=torch.float32, device="cuda") for _ in range(4)]
    kp = [t.data_ptr() for t in blk[:2]]
    vp = [t.data_ptr() for t in blk[2:]]
    L = fm.lib()

    def call(cache, count, first, span, pos_sum, newest, k=kp, v=vp):
        arr = lambda xs: (ctypes.c_int64 * max(len(xs), 1))(*xs)
        ptrs = lambda xs: (ctypes.c_void_p * max(len(xs), 1))(*xs)
        return L.fademem_set_state(ctypes.c_void_p(cache.handle), count, arr(first), arr(span), arr(pos_sum),
                                   newest, ptrs(k), ptrs(v), None)

    assert call(a, 5, [0] * 5, [1] * 5, [0] * 5, 9) == fm.FADEMEM_EINVAL           # count > M
    assert call(a, 2, [0, 0], [1, 1], [0, 0], 3) == fm.FADEMEM_EINVAL              # first not increasing
    assert call(a, 2, [0, 2], [3, 1], [3, 2], 3) == fm.FADEMEM_EINVAL              # overlaps the next entry
    assert call(a, 2, [0, 2], [0, 1], [0, 2], 3) == fm.FADEMEM_EINVAL              # span < 1
    assert call(a, 2, [0, 2], [2, 1], [9, 2], 3) == fm.FADEMEM_EINVAL              # pos_sum > newest * span
    assert call(a, 2, [0, 2], [2, 1], [1, 2], 1) == fm.FADEMEM_EINVAL              # newest below the last position
    assert call(a, 2, [0, 2], [2, 1], [1, 2], 3, k=[kp[0], 0]) == fm.FADEMEM_EINVAL  # NULL K
    assert a.count() == 0
    assert call(a, 0, [], [], [], 0) == fm.FADEMEM_OK and a.count() == 0          # empty snapshot: no-op
    assert call(a, 2, [0, 2], [2, 1], [1, 2], 3) == fm.FADEMEM_OK
    st = a.state()
    assert st == {"count": 2, "first": [0, 2], "span": [2, 1], "pos_sum": [1, 2], "newest": 3}
    assert call(a, 2, [0, 2], [2, 1], [1, 2], 3) == fm.FADEMEM_ESTATE             # no longer empty
