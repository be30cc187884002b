"""Build a copy of libfinemoe_map.so whose host code runs under AddressSanitizer
and UndefinedBehaviorSanitizer, for the CPU tests of the C ABI.

    python paper_2502_05370_amd/build_sanitized.py

Device code is compiled as in build.py (GPU sanitizers are not used: every
sanitizer option applies to the host pass only).  Objects go to
``_build_san/`` next to this file, the library to
``_build_san/libfinemoe_map_san.so``; the package loads it instead of the
regular library when FM_LIBRARY names it, with the sanitizer runtime
(sanitizer_runtime()) preloaded into the Python process.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)
import build as B  # noqa: E402

BUILD_DIR = os.path.join(HERE, "_build_san")
OUT = os.path.join(BUILD_DIR, "libfinemoe_map_san.so")

# host-pass only: each option right after -Xarch_host
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
            "-Xarch_host", "-shared-libasan"]


def sanitizer_runtime() -> str:
    """The shared ASan runtime of hipcc's clang (to preload into python)."""
    cands = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not cands:
        raise RuntimeError("the clang ASan runtime (libclang_rt.asan-x86_64.so) was not found")
    return cands[-1]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    common = [f for f in B.COMMON if f != "-O3"] + ["-O1", "-g"]
    cmd = [B.hipcc()] + lang + common + B.DEVICE_FLAGS + HOST_SAN + ["-c", os.path.join(B.CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        errs = "\n".join(l for l in (r.stderr or "").splitlines() if "packed-fp32-ops" not in l)
        raise RuntimeError(f"hipcc failed for {src}:\n{errs}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(B.SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, B.SOURCES))
    tmp = OUT + ".tmp"
    cmd = [B.hipcc(), "-shared", f"--offload-arch={B.ARCH}", "-fPIC"] + HOST_SAN + ["-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, OUT)
    if verbose:
        print(f"built {OUT}")
    return OUT


if __name__ == "__main__":
    build(verbose=True)
