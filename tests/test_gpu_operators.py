"""GPU parity of the consolidation operators of the ablation (Sec. 4.3
"Memory consolidation operator", Table 4): unweighted average, Select
Nearest and max pooling next to the sqrt-span default.

Same chunk loop as the other parity tests: attention over [memory || chunk],
then one Alg. S1 update per frame.  Schedule state, merge log and every
stored K/V entry are compared bit for bit with the oracle configured with
the same operator; attention within the bf16 / fp32 bars."""
import numpy as np
import pytest

from oracle import OracleCache
from paper_2606_10671_amd.synth import NumpyWanStream

from parity import check_attention, check_entries, check_state, oracle_attend, to_np

pytestmark = pytest.mark.gpu


def run(operator, dtype, H=2, D=64, N=80, F=2, M=5, chunks=14, anchor=True, layers=2, seed=3):
    import torch
    from paper_2606_10671_amd.fademem import Cache
    print(f"operator={operator} dtype={dtype} H={H} D={D} N={N} F={F} M={M} anchor={anchor} layers={layers}",
          flush=True)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=0.3, anchor=anchor, dtype=td,
                  layers=layers, merge_op=operator)
    ocs = [OracleCache(budget=M, beta=0.3, anchor=anchor, storage=dtype, operator=operator) for _ in range(layers)]
    streams = [NumpyWanStream(seed + 7 * l, N, H, D) for l in range(layers)]
    for c in range(chunks):
        frames = [[s.frame() for _ in range(F)] for s in streams]
        for l in range(layers):
            q = streams[l].queries(F * N)
            K = np.concatenate([f[0] for f in frames[l]])
            V = np.concatenate([f[1] for f in frames[l]])
            qd, kd, vd = (torch.from_numpy(np.ascontiguousarray(x)).to("cuda", td) for x in (q, K, V))
            lse = torch.empty((H, F * N), dtype=torch.float32, device="cuda")
            out = cache.attend(qd, kd, vd, layer=l, lse=lse)
            O_ref, L_ref = oracle_attend(ocs[l], q, K, V)
            check_attention(to_np(out), to_np(lse), O_ref, L_ref, dtype, where=(operator, c, l))
        for f in range(F):
            kf = [torch.from_numpy(frames[l][f][0]).to("cuda", td) for l in range(layers)]
            vf = [torch.from_numpy(frames[l][f][1]).to("cuda", td) for l in range(layers)]
            cache.insert(kf, vf, c * F + f)
            cache.consolidate()
            for l in range(layers):
                ocs[l].update(frames[l][f][0], frames[l][f][1], c * F + f)
        check_state(cache, ocs[0], where=(operator, c))
        for l in range(layers):
            check_entries(cache, ocs[l], layer=l, where=(operator, c, l))
    total, log = cache.merge_log()
    assert log == ocs[0].merge_log[-len(log):] and total == len(ocs[0].merge_log)
    return cache, ocs


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("operator", ["average", "select_nearest", "max"])
def test_operator_parity(operator, dtype):
    run(operator, dtype)


@pytest.mark.parametrize("operator", ["average", "select_nearest", "max"])
def test_operator_parity_d128_no_anchor(operator):
    """D = 128 (the attention kernel the benchmark times), anchor off so the first
    entry merges too."""
    run(operator, "bf16", H=3, D=128, N=70, F=3, M=4, chunks=10, anchor=False, layers=1)


def test_select_nearest_moves_no_bytes():
    """Select Nearest re-points the merged entry to the newer entry's slot:
    after a merge, the merged entry's K/V pointers are the ones the newer
    entry had, and the older entry's slot is the free one."""
    import torch
    from paper_2606_10671_amd.fademem import Cache
    H, D, N = 1, 64, 16
    cache = Cache(budget=2, heads=H, head_dim=D, tokens_per_block=N, beta=0.5, anchor=False,
                  dtype=torch.bfloat16, merge_op="select_nearest")
    gen = NumpyWanStream(11, N, H, D)
    for t in range(3):
        k, v = gen.frame()
        cache.insert(torch.from_numpy(k).to("cuda", torch.bfloat16), torch.from_numpy(v).to("cuda", torch.bfloat16), t)
    before = [cache.entry_kv(0, i) for i in range(3)]
    ptrs = [(k.data_ptr(), v.data_ptr()) for k, v in before]
    cache.consolidate()                        # the first merge at t = M picks pair 0
    after = [(k.data_ptr(), v.data_ptr()) for k, v in (cache.entry_kv(0, i) for i in range(2))]
    assert after[0] == ptrs[1] and after[1] == ptrs[2]
