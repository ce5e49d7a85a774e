#!/usr/bin/env python3
"""Benchmark of FadeMem's per-chunk cache step on one MI355X.

One step = one generated chunk: attention of the chunk's queries over
[memory || chunk] for every layer, then F x (insert + consolidate) -- the
hot path of the method (FadeMem Sec. 3.3, Alg. S1, Sec. 4.1).  Inputs are
seeded synthetic tensors already resident in HBM (no model weights exist
here); generation happens before the timed region.

Prints ONE JSON line (see the keys below).  Defaults: the Wan-1.3B-class
single-layer workload (12 heads x 128, 1560 tokens per latent frame,
3-frame chunks, budget 21, beta 0.3, anchor on, bf16).  Before the warm-up,
ceil(M/F) + 1 fill chunks bring the memory to its steady state (full, with
merges every frame), so every timed chunk attends over M*N + F*N keys and
runs F merges whatever --warmup says; then the warm-up chunks, untimed
settle chunks until the warm-up and settle chunks have lasted --settle
seconds (the chip's clock takes some tens of milliseconds of full load to
settle), and the timed chunks (8 warm-up and 104 timed by default, about 300
settle chunks at the default workload).  After the headline chunks, a 30-layer leg
times the chunk update alone (fused, then zero-copy staged), whose working
set is far above the 256 MB Infinity Cache: that is the merge's HBM
roofline figure.
"""
import argparse
import json
import math
import os
import sys
import time

WORKLOADS = {
    # name: heads, head_dim, tokens_per_block, frames_per_chunk, budget, layers, dtype, chunks (default run length)
    "wan1.3b-1layer": dict(heads=12, head_dim=128, tokens_per_block=1560, frames=3, budget=21, layers=1,
                           dtype="bf16", chunks=120),
    "wan1.3b-30layer": dict(heads=12, head_dim=128, tokens_per_block=1560, frames=3, budget=21, layers=30,
                            dtype="bf16", chunks=240),
    # about an hour of video at 16 fps with a 4x temporal VAE
    "wan1.3b-hour": dict(heads=12, head_dim=128, tokens_per_block=1560, frames=3, budget=21, layers=30,
                         dtype="bf16", chunks=4800),
    "wan14b-1layer": dict(heads=40, head_dim=128, tokens_per_block=3600, frames=3, budget=21, layers=1,
                          dtype="bf16", chunks=120),
    "wan14b-40layer": dict(heads=40, head_dim=128, tokens_per_block=3600, frames=3, budget=21, layers=40,
                           dtype="bf16", chunks=120),
    "tiny-fp32": dict(heads=2, head_dim=64, tokens_per_block=64, frames=1, budget=8, layers=1, dtype="f32",
                      chunks=40),
}
# The spectral-decay analysis (Sec. 3.2, S2) at the paper's scale: 374 clips of 177 latent frames of 60 x 104,
# every lag; a "step" is one analysis of all clips.
SPECTRAL = {"spectral-374clips": dict(clips=374, frames=177, height=60, width=104, bands=24, distinct=32)}

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
FP32_VECTOR_PEAK_TFLOPS = 157.3
FP32_MFMA_PEAK_TFLOPS = 157.3  # dense fp32 matrix-core peak (same figure as the vector peak)

# HBM bytes of one steady-state bf16 attention call (main kernel + merge of
# split tiles) at the wan1.3b-1layer workload, from rocprofv3 FETCH_SIZE and
# WRITE_SIZE (see profiles/attend_bf16_wan1.3b_1layer.md), valid only for the
# kernel source they were taken on (first 16 hex digits of its sha256).
ATTN_TRAFFIC = {"source_sha256": "a3f76e85dfec4181", "workload": "wan1.3b-1layer", "bytes_per_call": 1034552248}


# HBM bytes of one fused chunk update's data pass (update_data_kernel) in
# the 30-layer update leg, from rocprofv3 FETCH_SIZE and WRITE_SIZE scaled
# by the insert copy (see profiles/update_data_wan1.3b_30layer.md); valid
# only for the cache.hip source they were taken on.
UPD_TRAFFIC = {"source_sha256": "15da6713f8357ab0", "workload": "wan1.3b-30layer-update", "bytes_per_call": 4259822800}

# HBM bytes of one spectral analysis call (all its kernels) at spectral-374clips, from rocprofv3 FETCH_SIZE and
# WRITE_SIZE scaled by the insert copy (see profiles/spectral_fused_374clips.md); valid only for this source.
SPEC_TRAFFIC = {"source_sha256": "cdbe5ca3b4bd15d7", "workload": "spectral-374clips", "bytes_per_call": 1740286899}


def measured_traffic(table, source, workload):
    """Measured HBM bytes per call from `table`, or None if the kernel source
    changed since the counters were taken or the workload differs."""
    import hashlib
    src = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2606_10671_amd", "csrc", source)
    try:
        with open(src, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()[:16]
    except OSError:
        return None
    if table["source_sha256"] is None or sha != table["source_sha256"] or workload != table["workload"]:
        return None
    return table["bytes_per_call"]


def attn_traffic(workload):
    """Measured HBM bytes per attention call (None: source or workload differ)."""
    return measured_traffic(ATTN_TRAFFIC, "attend_bf16.hip", workload)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None,
                   help="timed chunks (default: the workload's chunk count minus the warm-up)")
    p.add_argument("--warmup", type=int, default=8)
    p.add_argument("--settle", type=float, default=0.3,
                   help="after the warm-up chunks, untimed chunks run until the load has lasted this many seconds")
    p.add_argument("--workload", default="wan1.3b-1layer", choices=sorted(WORKLOADS) + sorted(SPECTRAL))
    p.add_argument("--budget", type=int, default=None,
                   help="memory budget M in entries (default: the workload's; 12 is the paper's default, 15 slots with the current chunk)")
    p.add_argument("--beta", type=float, default=0.3)
    p.add_argument("--no-anchor", action="store_true")
    p.add_argument("--merge-op", default="sqrt_span", choices=["sqrt_span", "average", "select_nearest", "max"],
                   help="consolidation operator (Sec. 3.3 default, or a Table 4 ablation)")
    p.add_argument("--update", default="fused", choices=["fused", "single"],
                   help="fused: one fademem_update per chunk (the F updates in one pass); single: "
                        "fademem_insert + fademem_consolidate per frame")
    p.add_argument("--denoise-steps", type=int, default=1,
                   help="attention calls per layer per chunk (the generator's sampler calls it once per denoising "
                        "step on the same memory; the update follows the last step)")
    p.add_argument("--lse", action="store_true", help="have every attention call also return the log-sum-exp")
    p.add_argument("--rope-pairs", type=int, default=0,
                   help="temporal RoPE handling: pairs of each head carrying the temporal phase (Wan-class: 22 of "
                        "64); the memory is exposed re-indexed (0 = off)")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle CPU baseline")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-update-leg", action="store_true", help="skip the 30-layer chunk-update leg")
    p.add_argument("--update-leg-chunks", type=int, default=16, help="timed chunks of each update-leg mode")
    return p.parse_args()


def fused_block_ios(js, count0, F, M, anchor, merge_op, staged=False):
    """K (or V) block loads and stores of one fused chunk update, replayed
    from the merge decisions the library logged for it (no schedule
    arithmetic here): an operand is loaded once unless it is the result of
    an earlier merge of the same update; every new or changed entry is
    stored once, and a frame kept as is is also loaded once -- unless the
    frames are staged in pool slots (zero-copy), where a kept frame stays in
    its slot and moves no bytes."""
    refs = ["old"] * count0
    loads = 0
    it = iter(js)
    for _ in range(F):
        refs.append("old" if staged else "frame")
        if len(refs) > M:
            j = next(it)
            a, b = refs[j], refs[j + 1]
            if anchor and j == 0:
                new = a
            elif merge_op == "select_nearest":
                new = b
            else:
                loads += (a != "res") + (b != "res")
                new = "res"
            refs[j:j + 2] = [new]
    outs = [r for r in refs if r != "old"]
    return loads + outs.count("frame"), len(outs)


def cpu_baseline(wl, head_inputs, beta, anchor, budget_s, merge_op="sqrt_span"):
    """The oracle, as it stands, on the host cores: one steady-state chunk
    step (memory full, F merges) per head, heads taken in turn (and again,
    from a freshly filled memory, once all have run) until the time budget
    is spent, scaled to all heads and layers (the step is independent per
    head and per layer)."""
    from threadpoolctl import threadpool_info
    from oracle import OracleCache, chunk_step

    H, F = wl["heads"], wl["frames"]
    heads_done, t_total = 0, 0.0
    while t_total < budget_s:
        h = heads_done % H
        q, k, v, fill_k, fill_v = head_inputs(h)
        oc = OracleCache(budget=wl["budget"], beta=beta, anchor=anchor, storage=wl["dtype"], operator=merge_op)
        for t in range(len(fill_k)):          # fill the memory (untimed)
            oc.update(fill_k[t], fill_v[t], t)
        t0 = time.perf_counter()
        chunk_step(oc, q, k, v, F, len(fill_k))
        t_total += time.perf_counter() - t0
        heads_done += 1
    ms_chunk = t_total / heads_done * H * 1e3 * wl["layers"]
    blas_threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    return {
        "value": round(ms_chunk, 2), "unit": "ms/chunk", "cores": int(blas_threads), "kind": "oracle",
        "host_cpus": len(os.sched_getaffinity(0)),
        "sample": (f"one steady-state chunk step (fp64 attention over the full memory + {F} updates with "
                   f"merges) per head, {heads_done} head-steps of {H} heads of one layer, {t_total:.1f} s, "
                   f"scaled to {H} heads" + (f" x {wl['layers']} layers" if wl["layers"] > 1 else "")),
    }


def run_spectral(args):
    """Time the spectral-decay analysis (one library call per step)."""
    import torch
    from paper_2606_10671_amd import spectral as sp
    from paper_2606_10671_amd.synth import SpectralClips
    w = SPECTRAL[args.workload]
    C, T, H, W, K = w["clips"], w["frames"], w["height"], w["width"], w["bands"]
    steps = 10 if args.steps is None else args.steps
    dev = torch.device("cuda", 0)
    gen = SpectralClips(args.seed, T, H, W)  # generated on the host, then resident in HBM before timing
    distinct = [gen.clip() for _ in range(w["distinct"])]
    lat = torch.stack([distinct[c % len(distinct)] for c in range(C)]).to(dev).contiguous()
    band_np, centres = sp.radial_band_map(H, W, K)
    band = torch.from_numpy(band_np).to(dev)
    for _ in range(args.warmup):
        corr = sp.spectral_corr(lat, band, K, T - 1)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(steps):
        corr = sp.spectral_corr(lat, band, K, T - 1)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    h = sp.decorrelation_horizons(corr.cpu().numpy())
    ok = h > 0
    a, b = sp.fit_power_law(h[ok].astype(float), centres[ok]) if ok.sum() >= 2 else (None, None)
    flop = 2.0 * C * T * (H * W * W + H * H * W)  # the two contractions of every frame's DCT
    tflops = flop / (ms / 1e3) / 1e12
    # HBM: every latent frame read once (the transforms stay on chip), plus per-clip results (small)
    bytes_ = C * T * H * W * 4
    result = {
        "metric": "ms per spectral-decay analysis (DCT + band correlations over all clips)",
        "value": round(ms, 4), "unit": "ms/analysis", "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": f"synthetic multi-scale AR(1) latent clips ({w['distinct']} distinct, cycled)",
        "config": {"workload": args.workload, "clips": C, "frames": T, "height": H, "width": W, "bands": K,
                   "max_lag": T - 1},
        "dct_tflops": round(tflops, 3), "gbps": round(bytes_ / (ms / 1e3) / 1e9, 1),
        "fit": {"a": a, "b": b, "horizons": h.tolist()},
        "roofline": {"bound": "mfma", "kernel": "whole call (spectral_fused_kernel dominates)",
                     "achieved": round(tflops, 3), "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / FP32_MFMA_PEAK_TFLOPS, 4),
                     "traffic": measured_traffic(SPEC_TRAFFIC, "spectral.hip", args.workload),
                     "traffic_unit": "bytes per call (HBM read + write)"},
    }
    if not args.no_cpu_baseline:
        import oracle
        t0 = time.perf_counter()
        n = 0
        while n == 0 or (time.perf_counter() - t0 < args.cpu_seconds and n < C):
            oracle.band_correlations(distinct[n % len(distinct)][None].cpu().numpy(), band_np, K, T - 1)
            n += 1
        dt = time.perf_counter() - t0
        result["cpu_baseline"] = {"value": round(dt / n * C * 1e3, 1), "unit": "ms/analysis", "kind": "oracle",
                                  "cores": len(os.sched_getaffinity(0)),
                                  "sample": f"{n} of {C} clips, {dt:.1f} s, scaled to {C} clips"}
    print(json.dumps(result), flush=True)


def update_leg(args, M, anchor, L=30, H=12, D=128, N=1560, F=3):
    """The chunk update alone at the Wan-1.3B-class shape over L layers in
    one cache (working set ~6.9 GB, far above the 256 MB Infinity Cache):
    fill the memory, then time `--update-leg-chunks` fused updates
    (fademem_update: the caller's chunk is read, kept frames are copied into
    the pool) and as many zero-copy staged updates (fademem_update_staged:
    the chunk's frames are first written into the staging slots, as the
    model's K/V projection would, outside the timed calls).  One pair of
    events brackets the back-to-back fused updates, a pair each staged update
    call (the staging copies run between them); bytes are the algorithmic
    bytes replayed from the logged merge decisions."""
    import torch
    from paper_2606_10671_amd.fademem import Cache
    from paper_2606_10671_amd.synth import TorchWanStream
    dev = torch.device("cuda", 0)
    T = args.update_leg_chunks
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=args.beta, anchor=anchor,
                  dtype=torch.bfloat16, layers=L, device=dev, merge_op=args.merge_op, stage_frames=F)
    distinct = 4
    streams = [TorchWanStream(args.seed + 7000 + 1000 * l, N, H, D, device=dev) for l in range(L)]
    data = []
    for _ in range(distinct):
        per_layer = []
        for l in range(L):
            _, k, v = streams[l].chunk(F)
            per_layer.append((k.to(torch.bfloat16).contiguous(), v.to(torch.bfloat16).contiguous()))
        data.append(per_layer)
    stream = torch.cuda.current_stream()
    fill = -(-M // F) + 1
    c = 0
    for _ in range(fill):
        d = data[c % distinct]
        cache.update([x[0] for x in d], [x[1] for x in d], c * F)
        c += 1
    torch.cuda.synchronize()
    blk = N * H * D * 2
    modes = {}
    for mode in ("fused", "staged"):
        evs = []
        c0 = c
        if mode == "fused":
            # Back-to-back updates between one pair of events (each recorded
            # event leaves the GPU idle for a few microseconds).
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(T):
                d = data[c % distinct]
                cache.update([x[0] for x in d], [x[1] for x in d], c * F)
                c += 1
            e1.record(stream)
            evs.append((e0, e1))
        else:
            # The staging copies (the model's projection writing the frames)
            # run between the timed calls: a pair of events around each.
            for _ in range(T):
                d = data[c % distinct]
                slots = cache.stage(F)
                for l in range(L):
                    for f in range(F):
                        slots[l][f][0].copy_(d[l][0][f * N:(f + 1) * N])
                        slots[l][f][1].copy_(d[l][1][f * N:(f + 1) * N])
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                cache.update_staged(F, c * F)
                e1.record(stream)
                evs.append((e0, e1))
                c += 1
        torch.cuda.synchronize()
        ms_total = sum(a.elapsed_time(b) for a, b in evs)
        ms = [ms_total / T] * T
        _, log = cache.merge_log(cap=4096)
        js = log[len(log) - T * F:]
        bytes_ = 0
        for i in range(T):
            loads, stores = fused_block_ios(js[i * F:(i + 1) * F], M, F, M, anchor, args.merge_op,
                                            staged=(mode == "staged"))
            bytes_ += (loads + stores) * 2 * blk * L
        t_s = sum(ms) / 1e3
        modes[mode] = {"ms_per_update": round(sum(ms) / len(ms), 4),
                       "bytes_per_update": int(bytes_ // T),
                       "gbps": round(bytes_ / t_s / 1e9, 1) if bytes_ else None,
                       "first_chunk": c0, "chunks": T}
    cache.verify()
    del cache, data
    torch.cuda.empty_cache()
    fused = modes["fused"]
    traffic = measured_traffic(UPD_TRAFFIC, "cache.hip", "wan1.3b-30layer-update") if M == 21 else None
    roof = {"bound": "hbm", "kernel": f"update_plan_kernel + update_data_kernel (one fademem_update call, {L} layers)",
            "achieved": fused["gbps"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(fused["gbps"] / HBM_PEAK_GBS, 4) if fused["gbps"] else None,
            "traffic": traffic, "traffic_unit": "bytes per call (HBM read + write)",
            "algorithmic_bytes": fused["bytes_per_update"],
            "workload": f"wan1.3b-{L}layer-update (12x128 heads, 1560 tokens/frame, 3-frame chunks, budget {M})"}
    return roof, {"layers": L, **modes}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported by this build "
              "(the cache step shards by heads with no exchange, but no multi-GPU path is built).",
              file=sys.stderr)
        sys.exit(2)
    if args.workload in SPECTRAL:
        run_spectral(args)
        return
    import torch
    from paper_2606_10671_amd.fademem import Cache
    from paper_2606_10671_amd.synth import TorchWanStream

    wl = dict(WORKLOADS[args.workload])
    if args.budget is not None:
        if args.budget < 2:
            raise SystemExit("--budget must be at least 2 (one eligible pair besides the newest entry)")
        wl["budget"] = args.budget
    H, D, N, F, M, L = (wl[k] for k in ("heads", "head_dim", "tokens_per_block", "frames", "budget", "layers"))
    anchor = not args.no_anchor
    tdtype = torch.bfloat16 if wl["dtype"] == "bf16" else torch.float32
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    # Fill chunks: the memory holds M entries after ceil(M/F) chunks; one
    # more makes every later chunk's updates merge once per frame.
    fill = -(-M // F) + 1
    if args.steps is None:
        args.steps = max(1, wl["chunks"] - args.warmup - fill)
    chunks = fill + args.warmup + args.steps  # settle chunks are added below

    # ---- inputs, resident in HBM before timing -------------------------------
    # Distinct chunks are generated up to ~16 GB and then reused cyclically
    # (values do not change the work; the 1-layer workload keeps all 120).
    elt = 2 if tdtype == torch.bfloat16 else 4
    per_chunk_bytes = 3 * F * N * H * D * elt * L
    distinct = max(2, min(chunks, int(16e9 // per_chunk_bytes)))
    streams = [TorchWanStream(args.seed + 1000 * l, N, H, D, device=dev) for l in range(L)]
    inputs = []
    for c in range(distinct):
        per_layer = []
        for l in range(L):
            q, k, v = streams[l].chunk(F)
            per_layer.append((q.to(tdtype), k.to(tdtype).contiguous(), v.to(tdtype).contiguous()))
        inputs.append(per_layer)
    out = torch.empty((F * N, H, D), dtype=tdtype, device=dev)
    lse = torch.empty((H, F * N), dtype=torch.float32, device=dev) if args.lse else None
    cache = Cache(budget=M, heads=H, head_dim=D, tokens_per_block=N, beta=args.beta, anchor=anchor,
                  dtype=tdtype, layers=L, device=dev, merge_op=args.merge_op, rope_pairs=args.rope_pairs)
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    frame_elems = N * H * D

    def new_pair():
        return (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))

    def chunk_step(c, ev=None):
        per_layer = inputs[c % distinct]
        for _ in range(args.denoise_steps):
            for l in range(L):
                q, k, v = per_layer[l]
                if ev is not None:
                    ev["attn"].append(new_pair())
                    ev["attn"][-1][0].record(stream)
                    ev["keys"].append(cache.count() * N + F * N)  # host mirror of the count: no sync
                cache.attend(q, k, v, layer=l, out=out, lse=lse)
                if ev is not None:
                    ev["attn"][-1][1].record(stream)
        if args.update == "fused":
            cache.update([per_layer[l][1] for l in range(L)], [per_layer[l][2] for l in range(L)], c * F)
            return
        for f in range(F):
            ks = [per_layer[l][1][f * N:(f + 1) * N] for l in range(L)]
            vs = [per_layer[l][2][f * N:(f + 1) * N] for l in range(L)]
            if ev is not None:
                ev["ins"].append(new_pair())
                ev["ins"][-1][0].record(stream)
            cache.insert(ks, vs, c * F + f)
            if ev is not None:
                ev["ins"][-1][1].record(stream)
                ev["cons"].append(new_pair())
                ev["cons"][-1][0].record(stream)
            cache.consolidate()
            if ev is not None:
                ev["cons"][-1][1].record(stream)

    # Fill, warm-up, then settle chunks: the chip's clock takes some tens of
    # milliseconds of full load to settle (a kernel trace shows the first
    # attention calls over a full memory taking 1.17 ms, falling to 1.00 ms
    # over about 20 calls), so untimed chunks run until the warm-up and
    # settle chunks together have lasted --settle seconds, enqueued without
    # gaps (their count comes from the warm-up chunks' pace).
    for c in range(fill):
        chunk_step(c)
    torch.cuda.synchronize()
    t_w = time.time()
    warm = max(1, args.warmup)
    for c in range(fill, fill + warm):
        chunk_step(c)
    torch.cuda.synchronize()
    per_chunk_s = (time.time() - t_w) / warm
    settle = 0
    if per_chunk_s > 0 and args.settle > warm * per_chunk_s:
        settle = min(4096, int(math.ceil((args.settle - warm * per_chunk_s) / per_chunk_s)))
    for c in range(fill + warm, fill + warm + settle):
        chunk_step(c)
    torch.cuda.synchronize()
    first_timed = fill + warm + settle
    chunks = first_timed + args.steps
    merges_before, anchor_before = cache.merge_counts()

    # ---- timed region: whole chunk steps, with events around every attention
    # call on the stream the kernels run on (per-kernel averages come from
    # these).  Each recorded event leaves the GPU idle for a few microseconds,
    # so chunk and update times are read off the attention events instead of
    # events of their own: a chunk starts at its first attention call's start
    # event, and its update runs from its last attention call's end event to
    # the next chunk's start (so the update time includes the gaps of those
    # two events) ----------------------------------------------------------
    t_start, t_end = new_pair()
    ev = {"attn": [], "keys": [], "ins": [], "cons": []}
    torch.cuda.synchronize()
    t_start.record(stream)
    t_prog = time.time()
    for c in range(first_timed, chunks):
        chunk_step(c, ev)
        if time.time() - t_prog > 30:
            print(f"bench: chunk {c + 1}/{chunks} enqueued", file=sys.stderr, flush=True)
            t_prog = time.time()
    t_end.record(stream)
    torch.cuda.synchronize()
    ms_total = t_start.elapsed_time(t_end)
    ms_chunk = ms_total / args.steps
    calls = args.denoise_steps * L  # attention calls per chunk
    starts = [ev["attn"][i][0] for i in range(0, len(ev["attn"]), calls)] + [t_end]
    ends = [ev["attn"][i + calls - 1][1] for i in range(0, len(ev["attn"]), calls)]
    per_chunk = sorted(a.elapsed_time(b) for a, b in zip(starts[:-1], starts[1:]))
    ms_median = per_chunk[len(per_chunk) // 2]
    attn_ms = [a.elapsed_time(b) for a, b in ev["attn"]]
    ins_ms = [a.elapsed_time(b) for a, b in ev["ins"]]
    cons_ms = [a.elapsed_time(b) for a, b in ev["cons"]]
    upd_ms = [a.elapsed_time(b) for a, b in zip(ends, starts[1:])]
    cache_timed = cache

    total_merges, anchor_total = cache_timed.merge_counts()
    weighted = (total_merges - merges_before) - (anchor_total - anchor_before)
    blk = frame_elems * elt
    lk = M * N + F * N                      # keys per attention call at steady state
    assert all(k == lk for k in ev["keys"]), "a timed attention call saw a memory that is not full"
    attn_flop = sum(4.0 * (F * N) * k * D * H for k in ev["keys"])  # QK^T and PV of every timed call
    attn_avg_s = sum(attn_ms) / len(attn_ms) / 1e3
    attn_tflops = attn_flop / (sum(attn_ms) / 1e3) / 1e12
    # A weighted (or averaged, or max-pooled) merge reads two entries' K and V
    # and writes one; Select Nearest re-points a slot and moves no bytes.
    merge_bytes = 0 if args.merge_op == "select_nearest" else weighted * 3 * 2 * blk * L
    cons_s = sum(cons_ms) / 1e3
    merge_gbps = merge_bytes / cons_s / 1e9 if cons_s > 0 and merge_bytes > 0 else None
    ins_gbps = len(ins_ms) * 2 * 2 * blk * L / (sum(ins_ms) / 1e3) / 1e9 if ins_ms else None
    # Fused updates: algorithmic bytes from the logged merge decisions of the
    # timed chunks (the trailing chunks whose merges the log still holds).
    update_gbps = None
    if args.update == "fused":
        count, per_chunk_merges, count0s = 0, [], []
        for c in range(chunks):
            count0s.append(count)
            m = 0
            for _ in range(F):
                count += 1
                if count > M:
                    count -= 1
                    m += 1
            per_chunk_merges.append(m)
        _, log = cache_timed.merge_log(cap=4096)
        timed = list(range(first_timed, chunks))
        while timed and sum(per_chunk_merges[c] for c in timed) > len(log):
            timed.pop(0)
        js = log[len(log) - sum(per_chunk_merges[c] for c in timed):]
        bytes_, pos = 0, 0
        for c in timed:
            n = per_chunk_merges[c]
            loads, stores = fused_block_ios(js[pos:pos + n], count0s[c], F, M, anchor, args.merge_op)
            pos += n
            bytes_ += (loads + stores) * 2 * blk * L
        t_s = sum(upd_ms[c - first_timed] for c in timed) / 1e3
        update_gbps = bytes_ / t_s / 1e9 if t_s > 0 and bytes_ > 0 else None

    state = cache_timed.state()
    peak_bytes = cache_timed.pool_bytes
    is_bf16 = tdtype == torch.bfloat16
    peak = MFMA_BF16_PEAK_TFLOPS if is_bf16 else FP32_VECTOR_PEAK_TFLOPS
    result = {
        "metric": "ms per generated chunk (merge+attend), attention TFLOP/s, merge GB/s",
        "value": round(ms_chunk, 4),
        "unit": "ms/chunk",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_chunks": settle,
        "fill_chunks": fill,
        "ms_per_step": round(ms_chunk, 4),
        "ms_per_chunk_median": round(ms_median, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if is_bf16 else "f32",
        "data": "synthetic: seeded AR(1) K/V stream (rho 0.95, noise 0.5), N(0,1) Q, device-generated",
        "config": {"workload": args.workload, "heads": H, "head_dim": D, "tokens_per_block": N,
                   "frames_per_chunk": F, "query_tokens": F * N, "budget": M, "beta": args.beta,
                   "anchor": anchor, "merge_op": args.merge_op, "layers": L, "chunks": chunks,
                   "update": args.update, "denoise_steps": args.denoise_steps, "rope_pairs": args.rope_pairs,
                   "lse": args.lse, "keys_per_attend": lk},
        "attention_tflops": round(attn_tflops, 2),
        "attention_ms_per_call": round(attn_avg_s * 1e3, 4),
        "update": args.update,
        "denoise_steps": args.denoise_steps,
        "update_ms_per_chunk": round(sum(upd_ms) / len(upd_ms), 4),
        "update_gbps": round(update_gbps, 1) if update_gbps else None,
        "update_note": ("fused: algorithmic bytes of one pass (each operand block loaded once, each changed "
                        "entry stored once) / time from the chunk's last attention event to the next chunk's "
                        "first (plan + data kernels and the idle gaps of those two timing events)"
                        if args.update == "fused" else "single: F x (insert + consolidate) per chunk"),
        "merge_gbps": round(merge_gbps, 1) if merge_gbps else None,
        "merge_note": "single-frame path only: algorithmic bytes of weighted merges / time of consolidate calls",
        "weighted_merges_timed": weighted,
        "consolidate_ms_per_call": round(cons_s * 1e3 / len(cons_ms), 4) if cons_ms else None,
        "insert_gbps": round(ins_gbps, 1) if ins_gbps else None,
        "insert_ms_per_call": round(sum(ins_ms) / len(ins_ms), 4) if ins_ms else None,
        "pool_bytes": peak_bytes,
        "final_spans": state["span"],
        "roofline": {
            "bound": "mfma" if is_bf16 else "alu",
            "kernel": ("attend_bf16_d128 + attend_bf16_merge_d128 (one attend call)" if D == 128 else
                       "attend_bf16_d64 + attend_bf16_merge_d64 (one attend call)") if is_bf16
                      else "attend_f32_kernel + attend_f32_combine_kernel (one attend call)",
            "achieved": round(attn_tflops, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / peak, 4),
            "traffic": (attn_traffic(args.workload) if is_bf16 and M == WORKLOADS[args.workload]["budget"]
                        else None),
            "traffic_unit": "bytes per call (HBM read + write)",
        },
    }
    if not args.no_cpu_baseline:
        # The sample chunk follows exactly enough frames to fill the memory.
        c_fill = (M + F - 1) // F

        def head_inputs(h):
            def host(t):
                return t[:, h:h + 1].float().cpu().numpy()
            q, k, v = inputs[c_fill % distinct][0]
            fill_k, fill_v = [], []
            for c in range(c_fill):
                kc, vc = inputs[c % distinct][0][1], inputs[c % distinct][0][2]
                for f in range(F):
                    fill_k.append(host(kc[f * N:(f + 1) * N]))
                    fill_v.append(host(vc[f * N:(f + 1) * N]))
            return host(q), host(k), host(v), fill_k, fill_v
        result["cpu_baseline"] = cpu_baseline(wl, head_inputs, args.beta, anchor, args.cpu_seconds, args.merge_op)
    if not args.no_update_leg and args.workload.startswith("wan1.3b") and wl["dtype"] == "bf16":
        if L == 1:
            del inputs, cache, cache_timed
            torch.cuda.empty_cache()
            inputs = None
            result["merge_roofline"], result["update_leg"] = update_leg(args, M, anchor)
        elif update_gbps:
            result["merge_roofline"] = {
                "bound": "hbm", "kernel": f"update_plan_kernel + update_data_kernel (one fademem_update call, {L} layers)",
                "achieved": round(update_gbps, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(update_gbps / HBM_PEAK_GBS, 4), "traffic": None,
                "traffic_unit": "bytes per call (HBM read + write)", "workload": args.workload}
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
