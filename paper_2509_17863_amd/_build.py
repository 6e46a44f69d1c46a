"""Build libeaas.so (the HIP kernels + C ABI) in-tree for gfx950 with hipcc.

Beside the library, two copies whose grouped GEMMs use another tile
scheduler (EAAS_SCHEDULER 1 and 2 in csrc/gemm.hip) are linked for the
group-shrink ablation (bench.py --scheduler-ablation); nothing else loads
them."""
from __future__ import annotations

import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor
from pathlib import Path

PKG = Path(__file__).resolve().parent
CSRC = PKG / "csrc"
BUILD = PKG / "_build"
LIB = PKG / "libeaas.so"
SOURCES = ["route.hip", "gemm.hip", "combine.hip", "segments.hip", "quant.hip", "eaas_api.hip"]
# scheduler variants of the grouped GEMMs: library name -> EAAS_SCHEDULER
SCHEDULER_VARIANTS = {"scan_all": 1, "walk_all": 2}
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # keep the compiler from emitting packed fp32 vector ops on this target
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def variant_library(name: str) -> Path:
    """Path of a scheduler-variant library ("scan_all" or "walk_all")."""
    if name not in SCHEDULER_VARIANTS:
        raise ValueError(f"unknown scheduler variant {name!r}")
    return PKG / f"libeaas_sched_{name}.so"


def _compile(job) -> Path:
    src, suffix, defines = job
    obj = BUILD / (src.rsplit(".", 1)[0] + suffix + ".o")
    cmd = [hipcc(), *FLAGS, *defines, "-I", str(PKG.parent / "include"), "-c", str(CSRC / src),
           "-o", str(obj)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def _link(objs, out: Path) -> None:
    tmp = out.with_suffix(".so.tmp")
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *map(str, objs), "-o", str(tmp)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, out)


def build(jobs: int = 4) -> Path:
    """Compile every source and link libeaas.so and the scheduler variants;
    always rebuilds."""
    BUILD.mkdir(exist_ok=True)
    work = [(s, "", []) for s in SOURCES]
    work += [("gemm.hip", f"_sched{v}", [f"-DEAAS_SCHEDULER={v}"])
             for v in SCHEDULER_VARIANTS.values()]
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, work))
    base = objs[: len(SOURCES)]
    _link(base, LIB)
    gi = SOURCES.index("gemm.hip")
    for k, (name, v) in enumerate(SCHEDULER_VARIANTS.items()):
        objs_v = list(base)
        objs_v[gi] = objs[len(SOURCES) + k]
        _link(objs_v, variant_library(name))
    return LIB


if __name__ == "__main__":
    print(build())
