"""Build the plain C99 client of the C ABI (sf_c_client.c) with gcc, against
the in-tree libstagefrontier.so and the HIP runtime.  It is test
infrastructure: the GPU tests run it and compare its output with the oracle."""
from __future__ import annotations

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "sf_c_client.c")
OUT = os.path.join(HERE, "sf_c_client")
LIBDIR = os.path.join(ROOT, "paper_2606_06751_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(out: str = OUT) -> str:
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        raise FileNotFoundError("no C compiler (gcc) found")
    cmd = [cc, "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-isystem", os.path.join(ROCM, "include"),
           SRC, "-o", out + ".tmp",
           "-L", LIBDIR, "-lstagefrontier", "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           # the library is found next to the package wherever the tree is copied
           "-Wl,-rpath,$ORIGIN/../../paper_2606_06751_amd", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    if proc.returncode != 0:
        raise RuntimeError("C client build failed: %s\n%s%s" % (" ".join(cmd), proc.stdout, proc.stderr))
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build())
