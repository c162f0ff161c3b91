"""Compile libgt.so (all HIP sources + the C ABI) for gfx950 with hipcc.

Run as ``python -m paper_2407_14106_amd.build``; the library lands next to this
file.  Every compile uses -O3, wave64 gfx950 code only, and disables the packed
fp32 instruction forms.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(os.path.dirname(HERE), "include")
LIB = os.path.join(HERE, "libgt.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-fPIC",
    "-std=c++17",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
    "-I", INCLUDE,
    "-I", CSRC,
]


def sources() -> list[str]:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


def _compile(src: str, obj: str) -> tuple[str, int, str]:
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC, *FLAGS, *lang, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    return src, r.returncode, (r.stdout + r.stderr)


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every source and link libgt.so; returns its path (raises on failure)."""
    srcs = sources()
    tmp = tempfile.mkdtemp(prefix="gt_build_")
    try:
        objs = [os.path.join(tmp, os.path.basename(s) + ".o") for s in srcs]
        jobs = jobs or min(len(srcs), max(1, min(16, os.cpu_count() or 1)))
        with ThreadPoolExecutor(jobs) as ex:
            results = list(ex.map(lambda a: _compile(*a), zip(srcs, objs)))
        bad = [r for r in results if r[1] != 0]
        for src, rc, out in results:
            if verbose or rc != 0:
                noise = [l for l in out.splitlines() if "packed-fp32-ops" not in l]
                if noise:
                    print(f"--- {os.path.basename(src)} (rc={rc})\n" + "\n".join(noise), file=sys.stderr)
        if bad:
            raise RuntimeError("hipcc failed for: " + ", ".join(os.path.basename(b[0]) for b in bad))
        out_tmp = LIB + ".tmp"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", out_tmp]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
        os.replace(out_tmp, LIB)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
