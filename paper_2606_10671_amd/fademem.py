"""Python binding of libfademem.so (the C ABI in include/fademem.h).

Argument marshalling only: every step of the cache step runs in the
library's HIP kernels.  The functions keep the C names; ``Cache`` is a thin
owner of a device pool and a handle for use with torch tensors.  If the
library is not built, loading fails loudly -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libfademem.so")

FADEMEM_OK = 0
FADEMEM_EINVAL = -1
FADEMEM_ESTATE = -2
FADEMEM_ENOMEM = -3
FADEMEM_EHIP = -4
FADEMEM_EUNSUPPORTED = -5
FADEMEM_EINTERNAL = -6
FADEMEM_ESCRATCH = -7
FADEMEM_F32 = 0
FADEMEM_BF16 = 1
FADEMEM_MERGE_SQRT_SPAN = 0
FADEMEM_MERGE_AVERAGE = 1
FADEMEM_MERGE_SELECT_NEAREST = 2
FADEMEM_MERGE_MAX = 3
MERGE_OPS = {"sqrt_span": FADEMEM_MERGE_SQRT_SPAN, "average": FADEMEM_MERGE_AVERAGE,
             "select_nearest": FADEMEM_MERGE_SELECT_NEAREST, "max": FADEMEM_MERGE_MAX}

EXPORTED = (
    "fademem_pool_bytes", "fademem_cache_create", "fademem_cache_destroy", "fademem_insert",
    "fademem_consolidate", "fademem_update", "fademem_attend", "fademem_count", "fademem_get_state",
    "fademem_entry_kv", "fademem_set_state", "fademem_merge_log", "fademem_merge_counts", "fademem_last_hip_error",
    "fademem_strerror", "fademem_spectral_workspace_bytes", "fademem_spectral_corr", "fademem_stage",
    "fademem_update_staged", "fademem_attend_staged", "fademem_verify", "fademem_spectral_band_map",
    "fademem_spectral_horizons", "fademem_spectral_fit", "fademem_spectral_corr_static",
)


class fademem_config(ctypes.Structure):
    _fields_ = [
        ("budget", ctypes.c_int64),
        ("heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("tokens_per_block", ctypes.c_int64),
        ("beta", ctypes.c_double),
        ("anchor", ctypes.c_int32),
        ("merge_op", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("layers", ctypes.c_int32),
        ("rope_pairs", ctypes.c_int32),
        ("rope_theta", ctypes.c_double),
        ("stage_frames", ctypes.c_int32),
    ]


class FademError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        msg = lib().fademem_strerror(code).decode() if _LIB is not None else str(code)
        super().__init__(f"{where}: {msg} ({code})")


_LIB = None


def _check_single_hip_runtime():
    """The library must share the HIP runtime torch loaded (one libamdhip64
    in the process), or streams and pointers would belong to different
    runtimes."""
    try:
        with open("/proc/self/maps") as f:
            paths = {ln.split()[-1] for ln in f if "libamdhip64" in ln}
    except OSError:
        return
    if len({os.path.realpath(p) for p in paths}) > 1:
        raise RuntimeError("two HIP runtimes are mapped: " + ", ".join(sorted(paths)))


def lib() -> ctypes.CDLL:
    """Load libfademem.so (torch first, so its HIP runtime is the one used)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2606_10671_amd.build`")
    import torch  # noqa: F401  (maps torch's HIP runtime before ours)
    L = ctypes.CDLL(LIB_PATH)
    c_void_p, c_int64, c_int32, c_int = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int
    P = ctypes.POINTER
    L.fademem_strerror.argtypes = [c_int]
    L.fademem_strerror.restype = ctypes.c_char_p
    L.fademem_pool_bytes.argtypes = [P(fademem_config), P(ctypes.c_size_t)]
    L.fademem_cache_create.argtypes = [P(fademem_config), c_void_p, ctypes.c_size_t, c_void_p, P(c_void_p)]
    L.fademem_cache_destroy.argtypes = [c_void_p]
    L.fademem_insert.argtypes = [c_void_p, P(c_void_p), P(c_void_p), c_int64, c_void_p]
    L.fademem_consolidate.argtypes = [c_void_p, c_void_p]
    L.fademem_update.argtypes = [c_void_p, P(c_void_p), P(c_void_p), c_int64, c_int64, c_void_p]
    L.fademem_attend.argtypes = [c_void_p, c_int32, c_void_p, c_int64, c_void_p, c_void_p, c_int64,
                                 ctypes.c_float, c_void_p, c_void_p, c_void_p]
    L.fademem_count.argtypes = [c_void_p, P(c_int64)]
    L.fademem_get_state.argtypes = [c_void_p, P(c_int64), P(c_int64), P(c_int64), P(c_int64), P(c_int64),
                                    c_void_p]
    L.fademem_entry_kv.argtypes = [c_void_p, c_int32, c_int64, P(c_void_p), P(c_void_p), c_void_p]
    L.fademem_set_state.argtypes = [c_void_p, c_int64, P(c_int64), P(c_int64), P(c_int64), c_int64, P(c_void_p),
                                    P(c_void_p), c_void_p]
    L.fademem_merge_log.argtypes = [c_void_p, P(c_int32), c_int64, P(c_int64), c_void_p]
    L.fademem_merge_counts.argtypes = [c_void_p, P(c_int64), P(c_int64), c_void_p]
    L.fademem_spectral_workspace_bytes.argtypes = [c_int64, c_int64, c_int32, c_int32, c_int32, c_int64,
                                                   P(ctypes.c_size_t)]
    L.fademem_spectral_corr.argtypes = [c_void_p, c_int64, c_int64, c_int32, c_int32, c_void_p, c_int32, c_int64,
                                        c_void_p, ctypes.c_size_t, c_void_p, c_void_p]
    L.fademem_stage.argtypes = [c_void_p, c_int64, P(c_void_p), P(c_void_p)]
    L.fademem_update_staged.argtypes = [c_void_p, c_int64, c_int64, c_void_p]
    L.fademem_attend_staged.argtypes = [c_void_p, c_int32, c_void_p, c_int64, c_int64, ctypes.c_float, c_void_p,
                                        c_void_p, c_void_p]
    L.fademem_verify.argtypes = [c_void_p, c_void_p]
    L.fademem_spectral_corr_static.argtypes = [c_void_p, c_int64, c_int64, c_int32, c_int32, c_void_p, c_int32,
                                               c_int64, c_void_p, c_void_p]
    L.fademem_spectral_band_map.argtypes = [c_int32, c_int32, c_int32, c_void_p, c_void_p]
    L.fademem_spectral_horizons.argtypes = [c_void_p, c_int32, c_int64, c_int32, ctypes.c_double, c_void_p]
    L.fademem_spectral_fit.argtypes = [c_void_p, c_void_p, c_int64, c_int32, P(ctypes.c_double),
                                       P(ctypes.c_double)]
    L.fademem_last_hip_error.argtypes = [c_void_p]
    for name in EXPORTED:
        if name != "fademem_strerror":
            getattr(L, name).restype = c_int
    _LIB = L
    _check_single_hip_runtime()
    return L


def _ok(rc: int, where: str) -> None:
    if rc != FADEMEM_OK:
        raise FademError(rc, where)


def make_config(budget: int, heads: int, head_dim: int, tokens_per_block: int, beta: float = 0.3,
                anchor: bool = True, dtype: int = FADEMEM_BF16, layers: int = 1,
                merge_op: int = FADEMEM_MERGE_SQRT_SPAN, rope_pairs: int = 0,
                rope_theta: float = 10000.0, stage_frames: int = 0) -> fademem_config:
    return fademem_config(budget=budget, heads=heads, head_dim=head_dim, tokens_per_block=tokens_per_block,
                          beta=beta, anchor=int(anchor), merge_op=merge_op, dtype=dtype, layers=layers,
                          rope_pairs=rope_pairs, rope_theta=rope_theta, stage_frames=stage_frames)


# -- the C calls, same names ---------------------------------------------------

def fademem_pool_bytes(cfg: fademem_config) -> int:
    n = ctypes.c_size_t(0)
    _ok(lib().fademem_pool_bytes(ctypes.byref(cfg), ctypes.byref(n)), "fademem_pool_bytes")
    return n.value


def fademem_cache_create(cfg: fademem_config, pool_ptr: int, pool_bytes: int, stream: int = 0) -> int:
    h = ctypes.c_void_p(0)
    _ok(lib().fademem_cache_create(ctypes.byref(cfg), ctypes.c_void_p(pool_ptr), pool_bytes,
                                   ctypes.c_void_p(stream), ctypes.byref(h)), "fademem_cache_create")
    return h.value


def fademem_cache_destroy(handle: int) -> None:
    _ok(lib().fademem_cache_destroy(ctypes.c_void_p(handle)), "fademem_cache_destroy")


def fademem_insert(handle: int, k_ptrs: Sequence[int], v_ptrs: Sequence[int], position: int,
                   stream: int = 0) -> None:
    n = len(k_ptrs)
    ka = (ctypes.c_void_p * n)(*k_ptrs)
    va = (ctypes.c_void_p * n)(*v_ptrs)
    _ok(lib().fademem_insert(ctypes.c_void_p(handle), ka, va, position, ctypes.c_void_p(stream)), "fademem_insert")


def fademem_consolidate(handle: int, stream: int = 0) -> None:
    _ok(lib().fademem_consolidate(ctypes.c_void_p(handle), ctypes.c_void_p(stream)), "fademem_consolidate")


def fademem_update(handle: int, k_ptrs: Sequence[int], v_ptrs: Sequence[int], frames: int, first_position: int,
                   stream: int = 0) -> None:
    n = len(k_ptrs)
    ka = (ctypes.c_void_p * n)(*k_ptrs)
    va = (ctypes.c_void_p * n)(*v_ptrs)
    _ok(lib().fademem_update(ctypes.c_void_p(handle), ka, va, frames, first_position, ctypes.c_void_p(stream)),
        "fademem_update")


def fademem_attend(handle: int, layer: int, q_ptr: int, q_tokens: int, k_cur_ptr: int, v_cur_ptr: int,
                   cur_tokens: int, scale: float, out_ptr: int, lse_ptr: int = 0, stream: int = 0) -> None:
    _ok(lib().fademem_attend(ctypes.c_void_p(handle), layer, ctypes.c_void_p(q_ptr), q_tokens,
                             ctypes.c_void_p(k_cur_ptr), ctypes.c_void_p(v_cur_ptr), cur_tokens,
                             ctypes.c_float(scale), ctypes.c_void_p(out_ptr), ctypes.c_void_p(lse_ptr),
                             ctypes.c_void_p(stream)), "fademem_attend")


def fademem_stage(handle: int, layers: int, frames: int):
    """Device addresses of the staging slots: ([k per (layer, frame)], [v ...]), layer-major."""
    n = layers * frames
    ka, va = (ctypes.c_void_p * n)(), (ctypes.c_void_p * n)()
    _ok(lib().fademem_stage(ctypes.c_void_p(handle), frames, ka, va), "fademem_stage")
    return [int(x) for x in ka], [int(x) for x in va]


def fademem_update_staged(handle: int, frames: int, first_position: int, stream: int = 0) -> None:
    _ok(lib().fademem_update_staged(ctypes.c_void_p(handle), frames, first_position, ctypes.c_void_p(stream)),
        "fademem_update_staged")


def fademem_attend_staged(handle: int, layer: int, q_ptr: int, q_tokens: int, frames: int, scale: float,
                          out_ptr: int, lse_ptr: int = 0, stream: int = 0) -> None:
    _ok(lib().fademem_attend_staged(ctypes.c_void_p(handle), layer, ctypes.c_void_p(q_ptr), q_tokens, frames,
                                    ctypes.c_float(scale), ctypes.c_void_p(out_ptr), ctypes.c_void_p(lse_ptr),
                                    ctypes.c_void_p(stream)), "fademem_attend_staged")


def fademem_verify(handle: int, stream: int = 0) -> None:
    _ok(lib().fademem_verify(ctypes.c_void_p(handle), ctypes.c_void_p(stream)), "fademem_verify")


def fademem_count(handle: int) -> int:
    n = ctypes.c_int64(0)
    _ok(lib().fademem_count(ctypes.c_void_p(handle), ctypes.byref(n)), "fademem_count")
    return n.value


def fademem_get_state(handle: int, budget: int, stream: int = 0) -> dict:
    cap = budget + 1
    count, newest = ctypes.c_int64(0), ctypes.c_int64(0)
    first, span, pos_sum = (ctypes.c_int64 * cap)(), (ctypes.c_int64 * cap)(), (ctypes.c_int64 * cap)()
    _ok(lib().fademem_get_state(ctypes.c_void_p(handle), ctypes.byref(count), first, span, pos_sum,
                                ctypes.byref(newest), ctypes.c_void_p(stream)), "fademem_get_state")
    n = count.value
    return {"count": n, "first": list(first[:n]), "span": list(span[:n]), "pos_sum": list(pos_sum[:n]),
            "newest": newest.value}


def fademem_entry_kv(handle: int, layer: int, i: int, stream: int = 0):
    k, v = ctypes.c_void_p(0), ctypes.c_void_p(0)
    _ok(lib().fademem_entry_kv(ctypes.c_void_p(handle), layer, i, ctypes.byref(k), ctypes.byref(v),
                               ctypes.c_void_p(stream)), "fademem_entry_kv")
    return k.value, v.value


def fademem_set_state(handle: int, count: int, first: Sequence[int], span: Sequence[int], pos_sum: Sequence[int],
                      newest: int, k_ptrs: Sequence[int], v_ptrs: Sequence[int], stream: int = 0) -> None:
    n = max(count, 1)
    arr = lambda xs: (ctypes.c_int64 * n)(*xs)
    ptrs = lambda xs: (ctypes.c_void_p * max(len(xs), 1))(*xs)
    _ok(lib().fademem_set_state(ctypes.c_void_p(handle), count, arr(first), arr(span), arr(pos_sum), newest,
                                ptrs(k_ptrs), ptrs(v_ptrs), ctypes.c_void_p(stream)), "fademem_set_state")


def fademem_merge_log(handle: int, cap: int = 4096, stream: int = 0):
    buf = (ctypes.c_int32 * max(cap, 1))()
    total = ctypes.c_int64(0)
    _ok(lib().fademem_merge_log(ctypes.c_void_p(handle), buf, cap, ctypes.byref(total), ctypes.c_void_p(stream)),
        "fademem_merge_log")
    keep = min(total.value, cap, 4096)
    return total.value, list(buf[:keep])


def fademem_merge_counts(handle: int, stream: int = 0):
    """(total consolidations run, anchor merges among them)."""
    total, anchor = ctypes.c_int64(0), ctypes.c_int64(0)
    _ok(lib().fademem_merge_counts(ctypes.c_void_p(handle), ctypes.byref(total), ctypes.byref(anchor),
                                   ctypes.c_void_p(stream)), "fademem_merge_counts")
    return total.value, anchor.value


def fademem_spectral_workspace_bytes(clips: int, frames: int, height: int, width: int, bands: int,
                                     max_lag: int) -> int:
    n = ctypes.c_size_t(0)
    _ok(lib().fademem_spectral_workspace_bytes(clips, frames, height, width, bands, max_lag, ctypes.byref(n)),
        "fademem_spectral_workspace_bytes")
    return n.value


def fademem_spectral_corr(latents_ptr: int, clips: int, frames: int, height: int, width: int, band_of_ptr: int,
                          bands: int, max_lag: int, workspace_ptr: int, workspace_bytes: int, corr_ptr: int,
                          stream: int = 0) -> None:
    _ok(lib().fademem_spectral_corr(ctypes.c_void_p(latents_ptr), clips, frames, height, width,
                                    ctypes.c_void_p(band_of_ptr), bands, max_lag, ctypes.c_void_p(workspace_ptr),
                                    workspace_bytes, ctypes.c_void_p(corr_ptr), ctypes.c_void_p(stream)),
        "fademem_spectral_corr")


def fademem_spectral_corr_static(latents_ptr: int, clips: int, frames: int, height: int, width: int,
                                 band_of_ptr: int, bands: int, max_lag: int, corr_ptr: int, stream: int = 0) -> None:
    _ok(lib().fademem_spectral_corr_static(ctypes.c_void_p(latents_ptr), clips, frames, height, width,
                                           ctypes.c_void_p(band_of_ptr), bands, max_lag, ctypes.c_void_p(corr_ptr),
                                           ctypes.c_void_p(stream)), "fademem_spectral_corr_static")


def fademem_spectral_band_map(height: int, width: int, bands: int, band_of_ptr: int, centres_ptr: int = 0) -> None:
    _ok(lib().fademem_spectral_band_map(height, width, bands, ctypes.c_void_p(band_of_ptr),
                                        ctypes.c_void_p(centres_ptr)), "fademem_spectral_band_map")


def fademem_spectral_horizons(corr_ptr: int, bands: int, lags: int, window: int, drop: float,
                              horizon_ptr: int) -> None:
    _ok(lib().fademem_spectral_horizons(ctypes.c_void_p(corr_ptr), bands, lags, window, drop,
                                        ctypes.c_void_p(horizon_ptr)), "fademem_spectral_horizons")


def fademem_spectral_fit(t_ptr: int, r_ptr: int, n: int, iters: int = 100):
    a, b = ctypes.c_double(0.0), ctypes.c_double(0.0)
    _ok(lib().fademem_spectral_fit(ctypes.c_void_p(t_ptr), ctypes.c_void_p(r_ptr), n, iters, ctypes.byref(a),
                                   ctypes.byref(b)), "fademem_spectral_fit")
    return a.value, b.value


def fademem_last_hip_error(handle: int) -> int:
    return lib().fademem_last_hip_error(ctypes.c_void_p(handle))


def fademem_strerror(code: int) -> str:
    return lib().fademem_strerror(code).decode()


# -- torch-facing owner ----------------------------------------------------------

class Cache:
    """Owns a device pool (a torch uint8 tensor) and a library handle.

    Tensors are token-major [tokens][heads][head_dim], contiguous, on the
    current device, in the configured dtype (torch.float32 / torch.bfloat16).
    All calls enqueue on torch's current stream unless one is given.
    """

    def __init__(self, budget: int, heads: int, head_dim: int, tokens_per_block: int, beta: float = 0.3,
                 anchor: bool = True, dtype=None, layers: int = 1, device=None, merge_op: str = "sqrt_span",
                 rope_pairs: int = 0, rope_theta: float = 10000.0, stage_frames: int = 0):
        import torch
        dtype = torch.bfloat16 if dtype is None else dtype
        if dtype not in (torch.float32, torch.bfloat16):
            raise ValueError("dtype must be torch.float32 or torch.bfloat16")
        if merge_op not in MERGE_OPS:
            raise ValueError(f"merge_op must be one of {sorted(MERGE_OPS)}")
        self.torch_dtype = dtype
        self.cfg = make_config(budget, heads, head_dim, tokens_per_block, beta, anchor,
                               FADEMEM_BF16 if dtype == torch.bfloat16 else FADEMEM_F32, layers,
                               merge_op=MERGE_OPS[merge_op], rope_pairs=rope_pairs, rope_theta=rope_theta,
                               stage_frames=stage_frames)
        self.device = torch.device("cuda") if device is None else torch.device(device)
        self.pool_bytes = fademem_pool_bytes(self.cfg)
        self.pool = torch.empty(self.pool_bytes, dtype=torch.uint8, device=self.device)
        self.handle = fademem_cache_create(self.cfg, self.pool.data_ptr(), self.pool_bytes, self._stream(None))

    @staticmethod
    def _stream(stream) -> int:
        import torch
        s = torch.cuda.current_stream() if stream is None else stream
        return int(s.cuda_stream)

    def _check(self, t, rows: Optional[int] = None, name: str = "tensor"):
        if t.dtype != self.torch_dtype or not t.is_contiguous() or t.device.type != "cuda":
            raise ValueError(f"{name}: expected a contiguous {self.torch_dtype} CUDA tensor")
        if t.dim() != 3 or t.shape[1] != self.cfg.heads or t.shape[2] != self.cfg.head_dim:
            raise ValueError(f"{name}: expected [tokens][{self.cfg.heads}][{self.cfg.head_dim}]")
        if rows is not None and t.shape[0] != rows:
            raise ValueError(f"{name}: expected {rows} tokens")

    def insert(self, k, v, position: int, stream=None):
        ks = k if isinstance(k, (list, tuple)) else [k]
        vs = v if isinstance(v, (list, tuple)) else [v]
        if len(ks) != self.cfg.layers or len(vs) != self.cfg.layers:
            raise ValueError("one K and one V block per layer")
        for t in list(ks) + list(vs):
            self._check(t, self.cfg.tokens_per_block, "block")
        fademem_insert(self.handle, [t.data_ptr() for t in ks], [t.data_ptr() for t in vs], position,
                       self._stream(stream))

    def consolidate(self, stream=None):
        fademem_consolidate(self.handle, self._stream(stream))

    def update(self, k, v, first_position: int, stream=None):
        """A chunk's F updates (insert + consolidate per frame) in one call;
        k, v: per layer a [F*N][H][D] tensor (or one tensor for one layer)."""
        ks = k if isinstance(k, (list, tuple)) else [k]
        vs = v if isinstance(v, (list, tuple)) else [v]
        if len(ks) != self.cfg.layers or len(vs) != self.cfg.layers:
            raise ValueError("one K and one V chunk per layer")
        N = self.cfg.tokens_per_block
        rows = ks[0].shape[0] if ks[0].dim() == 3 else -1
        if rows <= 0 or rows % N:
            raise ValueError(f"chunk rows must be a positive multiple of {N}")
        for t in list(ks) + list(vs):
            self._check(t, rows, "chunk")
        fademem_update(self.handle, [t.data_ptr() for t in ks], [t.data_ptr() for t in vs], rows // N,
                       first_position, self._stream(stream))

    def attend(self, q, k_cur, v_cur, layer: int = 0, scale: float = 0.0, out=None, lse=None, stream=None):
        import torch
        self._check(q, None, "q")
        self._check(k_cur, None, "k_cur")
        self._check(v_cur, k_cur.shape[0], "v_cur")
        if out is None:
            out = torch.empty_like(q)
        self._check(out, q.shape[0], "out")
        if lse is not None and (lse.dtype != torch.float32 or not lse.is_contiguous()
                                or tuple(lse.shape) != (self.cfg.heads, q.shape[0])):
            raise ValueError("lse: expected a contiguous float32 [heads][q_tokens] tensor")
        fademem_attend(self.handle, layer, q.data_ptr(), q.shape[0], k_cur.data_ptr(), v_cur.data_ptr(),
                       k_cur.shape[0], scale, out.data_ptr(), 0 if lse is None else lse.data_ptr(),
                       self._stream(stream))
        return out

    def _block_view(self, ptr: int):
        import torch
        base = self.pool.data_ptr()
        elt = 2 if self.torch_dtype == torch.bfloat16 else 4
        n = self.cfg.tokens_per_block * self.cfg.heads * self.cfg.head_dim
        shape = (self.cfg.tokens_per_block, self.cfg.heads, self.cfg.head_dim)
        return self.pool[ptr - base: ptr - base + n * elt].view(self.torch_dtype).view(shape)

    def stage(self, frames: int):
        """Staging blocks for the zero-copy update: per layer, a list of
        `frames` (K, V) [N][H][D] views of free pool slots to write the chunk's
        frames into (valid until the next update)."""
        kp, vp = fademem_stage(self.handle, self.cfg.layers, frames)
        return [[(self._block_view(kp[l * frames + f]), self._block_view(vp[l * frames + f]))
                 for f in range(frames)] for l in range(self.cfg.layers)]

    def update_staged(self, frames: int, first_position: int, stream=None):
        fademem_update_staged(self.handle, frames, first_position, self._stream(stream))

    def attend_staged(self, q, frames: int, layer: int = 0, scale: float = 0.0, out=None, lse=None, stream=None):
        """Attention over [memory || the staged frames]."""
        import torch
        self._check(q, None, "q")
        if out is None:
            out = torch.empty_like(q)
        self._check(out, q.shape[0], "out")
        if lse is not None and (lse.dtype != torch.float32 or not lse.is_contiguous()
                                or tuple(lse.shape) != (self.cfg.heads, q.shape[0])):
            raise ValueError("lse: expected a contiguous float32 [heads][q_tokens] tensor")
        fademem_attend_staged(self.handle, layer, q.data_ptr(), q.shape[0], frames, scale, out.data_ptr(),
                              0 if lse is None else lse.data_ptr(), self._stream(stream))
        return out

    def verify(self, stream=None):
        """Check the host replay of the memory against the device (synchronises)."""
        fademem_verify(self.handle, self._stream(stream))

    def count(self) -> int:
        return fademem_count(self.handle)

    def state(self, stream=None) -> dict:
        return fademem_get_state(self.handle, self.cfg.budget, self._stream(stream))

    def merge_log(self, cap: int = 4096, stream=None):
        return fademem_merge_log(self.handle, cap, self._stream(stream))

    def merge_counts(self, stream=None):
        return fademem_merge_counts(self.handle, self._stream(stream))

    def entry_kv(self, layer: int, i: int, stream=None):
        """Views of logical entry i's K and V (valid until the next update)."""
        import torch
        kp, vp = fademem_entry_kv(self.handle, layer, i, self._stream(stream))
        return self._block_view(kp), self._block_view(vp)

    def snapshot(self, stream=None) -> dict:
        """Checkpoint: the metadata and device copies of every entry's K and V
        (per layer, oldest first)."""
        st = self.state(stream)
        kv = [[tuple(t.clone() for t in self.entry_kv(l, i, stream)) for i in range(st["count"])]
              for l in range(self.cfg.layers)]
        return {**st, "kv": kv}

    def restore(self, snap: dict, stream=None):
        """Resume: put a snapshot of a cache with the same configuration into
        this one, which must hold nothing yet."""
        n = snap["count"]
        ks = [snap["kv"][l][i][0] for l in range(self.cfg.layers) for i in range(n)]
        vs = [snap["kv"][l][i][1] for l in range(self.cfg.layers) for i in range(n)]
        for t in ks + vs:
            self._check(t, self.cfg.tokens_per_block, "entry")
        fademem_set_state(self.handle, n, snap["first"], snap["span"], snap["pos_sum"], snap["newest"],
                          [t.data_ptr() for t in ks], [t.data_ptr() for t in vs], self._stream(stream))

    def close(self):
        if getattr(self, "handle", None):
            fademem_cache_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
