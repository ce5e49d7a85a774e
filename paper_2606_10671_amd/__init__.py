"""FadeMem per-chunk cache step on MI355X (gfx950): HIP kernels behind the
C ABI of include/fademem.h, with a ctypes binding (``fademem``) and seeded
synthetic inputs (``synth``).  Importing the package loads nothing; the
library is loaded on first use of ``fademem``."""
__all__ = ["fademem", "synth", "build"]
