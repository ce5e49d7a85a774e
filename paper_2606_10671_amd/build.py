"""Build libfademem.so (all HIP sources, gfx950) in the package directory.

Usage: python -m paper_2606_10671_amd.build [-v] [--asan OUT]

--asan OUT builds the library with AddressSanitizer on its host code only
(the device code is unchanged) into OUT, for checking the host-side
validation.  To use it, copy OUT over the package's libfademem.so and run
with the clang ASan runtime preloaded, e.g.
LD_PRELOAD=<llvm>/lib/clang/<v>/lib/linux/libclang_rt.asan-x86_64.so
ASAN_OPTIONS=detect_leaks=0; build again without --asan afterwards.
"""
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libfademem.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # Keep the compiler from emitting packed fp32 ops (v_pk_*_f32).
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


def sources():
    return sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")))


ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer", "-shared-libsan", "-g"]


def build(verbose: bool = False, extra_flags=None, out: str = LIB) -> str:
    """Compile every HIP source into one shared library; returns its path."""
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *(extra_flags or []), "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(PKG, "csrc"), *sources(), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    msgs = [ln for ln in (res.stdout + res.stderr).splitlines() if noise not in ln]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    if "--asan" in sys.argv:
        print(build(verbose="-v" in sys.argv, extra_flags=ASAN_FLAGS, out=sys.argv[sys.argv.index("--asan") + 1]))
    else:
        print(build(verbose="-v" in sys.argv))
