"""Build the gfx950 HIP library in-tree: paper_2104_05755_amd/libtpp_mi355x.so.

Every source compiles to its own object (in parallel, under paper_2104_05755_amd/_build/), then
one hipcc line links the shared library.
"""
from __future__ import annotations

import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libtpp_mi355x.so")
OBJDIR = os.path.join(PKG, "_build")
SOURCES = ["tpp_api.hip", "brgemm_kernels.hip", "brgemm_dl_kernels.hip", "reduce_kernels.hip",
           "transform_kernels.hip", "embedding_kernels.hip", "equation.hip"]
# brgemm_dl_inst.hip is compiled once per part: (object stem, preprocessor definitions)
DL_PARTS = [("dl_bk32", ["-DDL_BK32"])] + [
    (f"dl_t{t}_a{a}_b{b}", [f"-DDL_TILE={t}", f"-DDL_AT={a}", f"-DDL_BT={b}"])
    for t in (256, 128, 64) for a in (0, 1) for b in (0, 1)]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _jobs() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def build(verbose: bool = False, extra: list | None = None, out: str = LIB) -> str:
    """Compile every HIP source of the library for gfx950 and link the shared library at `out`
    (`extra`: more hipcc options for every source, e.g. -D settings of the kernels' tunables)."""
    os.makedirs(OBJDIR, exist_ok=True)
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG, "csrc")]
    tag = f".{os.getpid()}"

    def compile_one(job):
        src, stem, defs = job
        obj = os.path.join(OBJDIR, f"{stem}{tag}.o")
        cmd = [hipcc(), *HIPCC_FLAGS, *(extra or []), *defs, *inc, "-c",
               os.path.join(PKG, "csrc", src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        return src, obj, r

    jobs = [("brgemm_dl_inst.hip", stem, defs) for stem, defs in DL_PARTS]
    jobs += [(s, s[:-4], []) for s in SOURCES]
    with ThreadPoolExecutor(max_workers=_jobs()) as ex:
        results = list(ex.map(compile_one, jobs))
    objs = []
    try:
        for src, obj, r in results:
            if r.returncode != 0:
                raise RuntimeError(f"hipcc failed on {src} ({r.returncode}):\n{r.stderr[-6000:]}")
            if verbose and r.stderr.strip():
                print(r.stderr[-4000:])
            objs.append(obj)
        tmp = out + f".tmp{os.getpid()}"
        cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc link failed ({r.returncode}):\n{r.stderr[-6000:]}")
        os.replace(tmp, out)
    finally:
        for _, obj, _ in results:
            if os.path.exists(obj):
                os.remove(obj)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
