"""Host AddressSanitizer + UndefinedBehaviorSanitizer build of the library, for the CPU tests.

The host-side runtime (argument validation, the create-time dry pass, the schedulers,
the actor-critic agent) is compiled with ``-fsanitize=address,undefined`` for the host
pass only; device code is never instrumented.  The two kernel-only sources are linked
from the ordinary build's objects.  The result, ``_build/san/librafiki_ensemble_san.so``,
is loaded by pointing ``RAFIKI_LIBRARY`` at it with the clang ASan runtime preloaded
(``env_for``), since the Python interpreter itself is not instrumented.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess

from . import build as b

SAN_DIR = os.path.join(b.OBJ, "san")
SAN_LIB = os.path.join(SAN_DIR, "librafiki_ensemble_san.so")
HOST_SOURCES = ["runtime.hip", "greedy.cpp", "rl.cpp"]      # instrumented
KERNEL_SOURCES = ["conv_mfma.hip", "conv_direct.hip", "misc.hip", "fused_net.hip"]   # linked as built
SAN_FLAGS = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined".split()
HOST_DEBUG = "-Xarch_host -fno-omit-frame-pointer -Xarch_host -g".split()


def asan_runtime() -> str:
    rts = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rts:
        raise RuntimeError("clang ASan runtime not found under /opt/rocm/llvm")
    return rts[-1]


def _compile(src: str, flags) -> str:
    out = os.path.join(SAN_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [b.HIPCC] + b.FLAGS + flags + ["-c", os.path.join(b.SRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    return out


def build_sanitized() -> str:
    os.makedirs(SAN_DIR, exist_ok=True)
    jobs = [(s, SAN_FLAGS + HOST_DEBUG) for s in HOST_SOURCES]
    # kernel-only sources: reuse the ordinary objects when they are newer than their
    # source and every header
    headers = glob.glob(os.path.join(b.SRC, "*.h")) + glob.glob(os.path.join(b.ROOT, "include", "*.h"))
    objs = []
    for s in KERNEL_SOURCES:
        o = os.path.join(b.OBJ, os.path.splitext(s)[0] + ".o")
        newest = max(os.path.getmtime(p) for p in headers + [os.path.join(b.SRC, s)])
        if os.path.exists(o) and os.path.getmtime(o) >= newest:
            objs.append(o)
        else:
            jobs.append((s, []))
    with cf.ThreadPoolExecutor(max_workers=min(len(jobs), 4)) as ex:
        objs += list(ex.map(lambda j: _compile(*j), jobs))
    rt = asan_runtime()
    tmp = SAN_LIB + ".tmp"
    cmd = [b.HIPCC, "--offload-arch=gfx950", "-shared"] + SAN_FLAGS + ["-shared-libsan", "-Wl,-rpath," +
                                                                     os.path.dirname(rt), "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, SAN_LIB)
    return SAN_LIB


def env_for(lib: str = SAN_LIB) -> dict:
    env = dict(os.environ)
    env.update({"RAFIKI_LIBRARY": lib, "LD_PRELOAD": asan_runtime(),
                # the interpreter's own allocations are not ours to report
                "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:halt_on_error=1",
                "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"})
    return env


if __name__ == "__main__":
    print(build_sanitized())
