"""Build libstagefrontier.so (HIP, gfx950) in-tree with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
# one translation unit per hot-path row, plus the C-ABI strings
SOURCES = [os.path.join(CSRC, f) for f in (
    "frontier.hip", "window.hip", "evidence.hip", "lag.hip", "median.hip", "gain.hip",
    "ingest.hip", "route.hip", "calib.hip", "abi.hip")]
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libstagefrontier.so")
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise FileNotFoundError("hipcc not found (set HIPCC or install ROCm)")


FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall",
    # keep the compiler from forming packed fp32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def compile_command(src: str, obj: str) -> list[str]:
    return [hipcc()] + FLAGS + ["-I", INCLUDE, "-I", CSRC, "-c", src, "-o", obj]


def link_command(objs: list[str], out: str) -> list[str]:
    return [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC"] + objs + ["-o", out]


def _run(cmd):
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError("hipcc failed: %s\n%s%s" % (" ".join(cmd), proc.stdout, proc.stderr))


def build(out: str = LIB) -> str:
    """Compile every source in parallel, then link the shared library."""
    from concurrent.futures import ThreadPoolExecutor

    objdir = tempfile.mkdtemp(prefix="sf_build_")
    try:
        objs = [os.path.join(objdir, os.path.basename(src) + ".o") for src in SOURCES]
        with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
            list(ex.map(lambda so: _run(compile_command(*so)), zip(SOURCES, objs)))
        tmp = out + ".tmp%d" % os.getpid()
        _run(link_command(objs, tmp))
        os.replace(tmp, out)
    finally:
        shutil.rmtree(objdir, ignore_errors=True)
    return out


if __name__ == "__main__":
    print(build())
