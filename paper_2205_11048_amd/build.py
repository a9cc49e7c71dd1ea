"""Build the HIP libraries in-tree for gfx950.

``libgba.so`` (the push-step, from ``csrc/*.hip``) lands next to this file;
the synthetic-input generator (``synth/gen.hip``) is built into
``synth/libgba_synth.so``.  Run ``python -m paper_2205_11048_amd.build``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
ARCH = os.environ.get("GBA_OFFLOAD_ARCH", "gfx950")

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    # keep the compiler from emitting packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("build failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    return r


def build_shared(sources, out_so, include_dirs=(), jobs=8):
    build_dir = os.path.join(os.path.dirname(out_so), "_build")
    os.makedirs(build_dir, exist_ok=True)
    inc = [f"-I{d}" for d in include_dirs]

    def compile_one(src):
        obj = os.path.join(build_dir, os.path.splitext(os.path.basename(src))[0] + ".o")
        _run([HIPCC, *FLAGS, *inc, "-c", src, "-o", obj])
        return obj

    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(compile_one, sources))
    tmp = out_so + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, out_so)
    return out_so


def build_gba(jobs=8):
    csrc = os.path.join(PKG, "csrc")
    srcs = sorted(os.path.join(csrc, f) for f in os.listdir(csrc) if f.endswith(".hip"))
    return build_shared(srcs, os.path.join(PKG, "libgba.so"), [csrc, os.path.join(ROOT, "include")], jobs)


def build_synth(jobs=8):
    sdir = os.path.join(ROOT, "synth")
    return build_shared([os.path.join(sdir, "gen.hip")], os.path.join(sdir, "libgba_synth.so"), [sdir], jobs)


def build_all(jobs=8):
    return [build_gba(jobs), build_synth(jobs)]


def build_gba_host_sanitized(jobs=8):
    """libgba.so with AddressSanitizer and UndefinedBehaviorSanitizer on its
    host code only (argument checks, workspace layout, launch logic; device
    code is built as usual), into _build_sanitized/.  Load it by naming it in
    GBA_LIBRARY, with the clang AddressSanitizer runtime in LD_PRELOAD (its
    libclang_rt.asan-x86_64.so under /opt/rocm/llvm/lib/clang/*/lib/linux/),
    on a machine without a GPU: the host-path tests then run every entry
    point's checks and layout arithmetic under the sanitizers."""
    csrc = os.path.join(PKG, "csrc")
    srcs = sorted(os.path.join(csrc, f) for f in os.listdir(csrc) if f.endswith(".hip"))
    out_dir = os.path.join(PKG, "_build_sanitized")
    os.makedirs(out_dir, exist_ok=True)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
    inc = [f"-I{csrc}", f"-I{os.path.join(ROOT, 'include')}"]

    def compile_one(src):
        obj = os.path.join(out_dir, os.path.splitext(os.path.basename(src))[0] + ".o")
        _run([HIPCC, *FLAGS, *san, *inc, "-c", src, "-o", obj])
        return obj

    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(compile_one, srcs))
    out_so = os.path.join(out_dir, "libgba_sanitized.so")
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *san, *objs, "-o", out_so])
    return out_so


if __name__ == "__main__":
    if "--sanitize-host" in sys.argv:
        print("built", build_gba_host_sanitized())
        sys.exit(0)
    for p in build_all():
        print("built", p)
    sys.exit(0)
