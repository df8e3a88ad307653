"""Builds libpr2 with AddressSanitizer and UndefinedBehaviorSanitizer on its
HOST code, for CPU checks of the argument-validation layer.

The sanitizer flags go to the host compilation only (each behind
``-Xarch_host``); the device code is compiled as usual and not instrumented.
The library's C entry points, checks, workspace layouts and records are
instrumented.  Python loads it with the shared ASan runtime preloaded;
``runtime_preload()`` names that runtime.  Output: ``_build_san/libpr2_san.so``
next to this file, rebuilt only when a source or flag changed.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build_san")
LIB = os.path.join(BUILD, "libpr2_san.so")
HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/lib/llvm/bin/clang"
# each sanitizer flag goes to the host compilation only
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]
FLAGS = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-command-line-argument"] + SAN


def runtime_preload() -> str:
    """Path of the shared ASan runtime to preload into an uninstrumented python."""
    return subprocess.run([CLANG, "-print-file-name=libclang_rt.asan-x86_64.so"],
                          check=True, capture_output=True, text=True).stdout.strip()


def _stamp(sources) -> str:
    import hashlib
    h = hashlib.sha256(" ".join(FLAGS).encode())
    for name in sorted(os.listdir(CSRC)):
        h.update(name.encode())
        h.update(open(os.path.join(CSRC, name), "rb").read())
    h.update(open(os.path.join(HERE, "..", "include", "pr2.h"), "rb").read())
    h.update(" ".join(sources).encode())
    return h.hexdigest()


def build() -> str:
    from paper_2606_00395_amd.build import SOURCES
    os.makedirs(BUILD, exist_ok=True)
    stamp_path = os.path.join(BUILD, "stamp")
    stamp = _stamp(SOURCES)
    if os.path.exists(LIB) and os.path.exists(stamp_path) and open(stamp_path).read() == stamp:
        return LIB
    objs, cmds = [], []
    for src in SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        objs.append(obj)
        cmds.append([HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])

    def run(cmd):
        p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
        p.stdout = "\n".join(l for l in p.stdout.splitlines()
                             if "packed-fp32-ops' is not a recognized feature" not in l)
        return p
    with ThreadPoolExecutor(len(cmds)) as ex:
        for cmd, p in zip(cmds, ex.map(run, cmds)):
            if p.returncode != 0:
                print(p.stdout, file=sys.stderr)
                raise RuntimeError("hipcc failed: " + " ".join(cmd))
    p = run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-shared-libasan", *SAN, "-o",
             LIB, *objs])
    if p.returncode != 0:
        print(p.stdout, file=sys.stderr)
        raise RuntimeError("link failed")
    with open(stamp_path, "w") as f:
        f.write(stamp)
    return LIB


if __name__ == "__main__":
    print(build())
