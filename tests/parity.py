"""Shared helpers of the GPU parity tests: run the library and the oracle
on the same seeded inputs and compare element by element."""
import numpy as np

from oracle import OracleCache, attend

# Tolerances (stated by the acceptance bar of the cache step):
F32_NORM_RTOL = 1e-5    # fp32 attention, normwise relative
BF16_MAX_ABS = 2e-2     # bf16 attention, max abs vs the fp64 oracle
BF16_NORM_RTOL = 1e-2   # bf16 attention, normwise relative (diagnostic bar)
# bf16 attention, max abs LSE error (diagnostic bar: it catches a dropped or
# duplicated entry, which a max-abs bar on O near the output's own scale
# cannot).  The LSE comes from an fp32 sum of the unrounded softmax weights.
BF16_LSE_ABS = 2e-3
F32_LSE_ABS = 1e-5


def to_np(t):
    import torch
    return t.detach().to("cpu", torch.float32).numpy()


def check_state(cache, ocache: OracleCache, where=""):
    st = cache.state()
    ost = ocache.state()
    assert st["count"] == ost["count"], where
    assert st["first"] == ost["first"], where
    assert st["span"] == ost["span"], where
    assert st["pos_sum"] == ost["pos_sum"], where
    assert st["newest"] == ost["newest"], where


def check_entries(cache, ocache: OracleCache, layer=0, where="", head_slice=None):
    """Bitwise equality of every entry's stored K and V."""
    for i, e in enumerate(ocache.entries):
        k, v = cache.entry_kv(layer, i)
        kg, vg = to_np(k), to_np(v)
        if head_slice is not None:
            kg, vg = kg[:, head_slice], vg[:, head_slice]
        assert np.array_equal(kg.view(np.uint32), np.asarray(e.K, np.float32).view(np.uint32)), (where, "K", i)
        assert np.array_equal(vg.view(np.uint32), np.asarray(e.V, np.float32).view(np.uint32)), (where, "V", i)


def check_attention(O, LSE, O_ref, LSE_ref, dtype, where=""):
    """O, LSE from the GPU (numpy float32); O_ref, LSE_ref fp64 oracle."""
    err = np.abs(O.astype(np.float64) - O_ref)
    norm = np.linalg.norm(O.astype(np.float64) - O_ref) / max(np.linalg.norm(O_ref), 1e-300)
    lse_err = np.abs(LSE.astype(np.float64) - LSE_ref).max() if LSE is not None else 0.0
    if dtype == "f32":
        assert norm <= F32_NORM_RTOL, (where, norm)
        assert lse_err <= F32_LSE_ABS * max(1.0, np.abs(LSE_ref).max()), (where, lse_err)
    else:
        assert err.max() <= BF16_MAX_ABS, (where, err.max())
        assert norm <= BF16_NORM_RTOL, (where, norm)
        assert lse_err <= BF16_LSE_ABS, (where, lse_err)
    return float(err.max()), float(norm), float(lse_err)


def oracle_attend(ocache, Q, Kc, Vc, scale=None):
    Km, Vm = ocache.exposed_kv()
    return attend(Q, Km, Vm, Kc, Vc, scale=scale)
