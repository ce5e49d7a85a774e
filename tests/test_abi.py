"""Host-side checks of the C ABI that need no GPU: the library loads, it
exports every function include/fademem.h declares, and configuration /
argument validation rejects bad input before anything is enqueued."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2606_10671_amd import fademem as fm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fademem.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fademem_[a-z_]+)\s*\(", text)))


def test_header_declares_the_binding_surface():
    assert declared_functions() == sorted(fm.EXPORTED)


def test_library_exports_every_declared_symbol():
    assert os.path.exists(fm.LIB_PATH), "build the library first"
    out = subprocess.run(["nm", "-D", "--defined-only", fm.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if " T " in ln}
    for name in declared_functions():
        assert name in exported, name
    lib = fm.lib()
    for name in declared_functions():
        assert getattr(lib, name) is not None


def test_strerror_covers_all_codes():
    for code in (fm.FADEMEM_OK, fm.FADEMEM_EINVAL, fm.FADEMEM_ESTATE, fm.FADEMEM_ENOMEM, fm.FADEMEM_EHIP,
                 fm.FADEMEM_EUNSUPPORTED, fm.FADEMEM_EINTERNAL, fm.FADEMEM_ESCRATCH):
        assert fm.fademem_strerror(code) != "unknown error"
    assert fm.fademem_strerror(-99) == "unknown error"


GOOD = dict(budget=21, heads=12, head_dim=128, tokens_per_block=1560, beta=0.3, anchor=True,
            dtype=fm.FADEMEM_BF16, layers=1)


def test_pool_bytes_layout():
    """Metadata (< 64 KiB) + (M+1) K and V slots per layer; bf16 caches add
    the attention's split-work scratch: two slots per workgroup (at most
    256) of 256 queries x D fp32 partial O plus 1024 fp32 maxima and sums
    (the same bytes as 512 slots of 128 queries x D plus 512 floats); fp32
    caches add 512 slots of 64 queries x (D + 2) floats for key ranges."""
    n = fm.fademem_pool_bytes(fm.make_config(**GOOD))
    blk = 1560 * 12 * 128 * 2
    ws = 2 * 512 * (128 * 128 + 2 * 256) * 4
    assert n >= 22 * 2 * blk + ws and n < 22 * 2 * blk + ws + 64 * 1024
    n30 = fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "layers": 30}))
    assert n30 - n == 29 * 22 * 2 * blk
    nf = fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "dtype": fm.FADEMEM_F32}))
    assert nf - n == 22 * 2 * blk - ws + 512 * 64 * (128 + 2) * 4
    n64 = fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "head_dim": 64}))
    assert n - n64 == 22 * blk + ws - 2 * 512 * (128 * 64 + 2 * 256) * 4
    # staging three frames: M + 3 slots per layer instead of M + 1
    ns = fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "stage_frames": 3}))
    assert ns - n == 2 * 2 * blk
    assert fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "stage_frames": 1})) == n


def test_rope_view_covers_every_exposable_entry():
    """Temporal RoPE handling adds one re-indexed K block per slot and layer:
    the M + 1 entries held between an insert and its consolidation, or M
    plus the staged frames, all fit (a view of M blocks would overrun)."""
    n = fm.fademem_pool_bytes(fm.make_config(**GOOD))
    blk = 1560 * 12 * 128 * 2
    nr = fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "rope_pairs": 22}))
    assert 22 * blk <= nr - n < 22 * blk + 64 * 1024
    nr30 = fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "rope_pairs": 22, "layers": 30}))
    n30 = fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "layers": 30}))
    assert 30 * 22 * blk <= nr30 - n30 < 30 * 22 * blk + 64 * 1024
    nrs = fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "rope_pairs": 22, "stage_frames": 3}))
    ns = fm.fademem_pool_bytes(fm.make_config(**{**GOOD, "stage_frames": 3}))
    assert 24 * blk <= nrs - ns < 24 * blk + 64 * 1024


@pytest.mark.parametrize("field,value", [("budget", 1), ("budget", 1024), ("heads", 0), ("head_dim", 96),
                                         ("tokens_per_block", 0), ("beta", 0.0), ("beta", 1.0001),
                                         ("beta", float("nan")), ("anchor", 2), ("dtype", 7), ("layers", 0),
                                         ("merge_op", -1), ("merge_op", 4), ("rope_pairs", -1),
                                         ("rope_pairs", 65), ("rope_theta", 1.0), ("stage_frames", -1),
                                         ("stage_frames", 5)])
def test_bad_configs_are_rejected(field, value):
    cfg = fm.make_config(**GOOD)
    if field == "rope_theta":
        cfg.rope_pairs = 22
    setattr(cfg, field, value)
    with pytest.raises(fm.FademError) as e:
        fm.fademem_pool_bytes(cfg)
    assert e.value.code == fm.FADEMEM_EINVAL


def test_create_validates_before_touching_the_device():
    cfg = fm.make_config(**GOOD)
    need = fm.fademem_pool_bytes(cfg)
    L = fm.lib()
    h = ctypes.c_void_p(0)
    assert L.fademem_cache_create(ctypes.byref(cfg), None, need, None, ctypes.byref(h)) == fm.FADEMEM_EINVAL
    assert L.fademem_cache_create(ctypes.byref(cfg), ctypes.c_void_p(4096 + 8), need, None,
                                  ctypes.byref(h)) == fm.FADEMEM_EINVAL           # misaligned
    assert L.fademem_cache_create(ctypes.byref(cfg), ctypes.c_void_p(4096), need - 1, None,
                                  ctypes.byref(h)) == fm.FADEMEM_ENOMEM
    cfg.merge_op = 4          # no such consolidation operator
    assert L.fademem_cache_create(ctypes.byref(cfg), ctypes.c_void_p(4096), need, None,
                                  ctypes.byref(h)) == fm.FADEMEM_EINVAL
    assert h.value is None
    assert L.fademem_cache_create(ctypes.byref(cfg), ctypes.c_void_p(4096), need, None, None) == fm.FADEMEM_EINVAL


def test_null_handles_are_rejected():
    L = fm.lib()
    assert L.fademem_consolidate(None, None) == fm.FADEMEM_EINVAL
    assert L.fademem_insert(None, None, None, 0, None) == fm.FADEMEM_EINVAL
    assert L.fademem_update(None, None, None, 3, 0, None) == fm.FADEMEM_EINVAL
    assert L.fademem_attend(None, 0, None, 1, None, None, 0, ctypes.c_float(0), None, None, None) == fm.FADEMEM_EINVAL
    assert L.fademem_stage(None, 1, None, None) == fm.FADEMEM_EINVAL
    assert L.fademem_update_staged(None, 1, 0, None) == fm.FADEMEM_EINVAL
    assert L.fademem_attend_staged(None, 0, None, 1, 1, ctypes.c_float(0), None, None, None) == fm.FADEMEM_EINVAL
    assert L.fademem_verify(None, None) == fm.FADEMEM_EINVAL
    n = ctypes.c_int64(0)
    assert L.fademem_count(None, ctypes.byref(n)) == fm.FADEMEM_EINVAL
    assert L.fademem_cache_destroy(None) == fm.FADEMEM_OK
