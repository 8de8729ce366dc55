"""Build the native libraries in-tree with hipcc for gfx950.

* ``libfff.so``      -- the product: the C ABI of include/fff.h over the HIP kernels.
* ``libfffbench.so`` -- benchmark-only helpers (dense FF comparator, copy kernel).

Usage: ``python -m paper_2311_10770_amd.build``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import time
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
INCLUDE = ROOT / "include"
BUILD = ROOT / "_build"

ARCH = "gfx950"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# -packed-fp32-ops: no v_pk_{add,mul,fma}_f32 in device code (it is a device
# feature; the host pass warns that it does not know it).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall", "-fvisibility=hidden",
          f"-I{INCLUDE}", f"-I{CSRC}"] + DEVICE_FLAGS

LIBS = {
    "libfff.so": {"sources": ["fff_api.cpp", "fff_kernels.hip", "fff_backward.hip", "fff_masked.hip", "fff_gemm.hip",
                              "fff_subtree.hip"],
                  "link": []},
    "libfffbench.so": {"sources": ["bench_helpers.hip"], "link": ["-L/opt/rocm/lib", "-lhipblaslt"]},
}


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(" ".join(cmd) + "\n" + r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd[-3:])}")
    return r


def _compile(src: Path, obj: Path):
    lang = ["-x", "hip"]
    _run([HIPCC, *COMMON, *lang, "-c", str(src), "-o", str(obj)])
    return obj


def build_lib(name: str, jobs: int = 4) -> Path:
    spec = LIBS[name]
    BUILD.mkdir(exist_ok=True)
    srcs = [CSRC / s for s in spec["sources"] if (CSRC / s).exists()]
    if not srcs:
        raise FileNotFoundError(f"no sources for {name}")
    objs = [BUILD / (s.stem + ".o") for s in srcs]
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        list(ex.map(_compile, srcs, objs))
    out = PKG / name
    tmp = out.with_suffix(".so.tmp")
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", str(tmp), *map(str, objs), *spec["link"]])
    os.replace(tmp, out)
    return out


def build_all(jobs: int = 4) -> list:
    if shutil.which(HIPCC) is None and not Path(HIPCC).exists():
        raise FileNotFoundError(f"hipcc not found at {HIPCC}")
    t0 = time.time()
    built = [build_lib(n, jobs) for n in LIBS if any((CSRC / s).exists() for s in LIBS[n]["sources"])]
    print(f"[build] {', '.join(p.name for p in built)} in {time.time() - t0:.1f}s", flush=True)
    return built


if __name__ == "__main__":
    build_all()
