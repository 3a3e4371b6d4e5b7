"""Build the HIP library in-tree for gfx950.

``python -m paper_2607_16100_amd.build`` compiles the kernels and the C ABI
into ``paper_2607_16100_amd/libllcoll.so`` with hipcc:

* ``csrc/ll_inst.hip`` once per rank count P = 2..8 (``-DLL_INST_P=P``): the
  kernel instantiations for that P;
* ``csrc/llcoll.hip``: the host entry points, the fill and probe kernels;

each to an object of its own, in parallel, then linked into one shared
library.  Extra preprocessor definitions (diagnostic builds) can be passed
with ``extra_defines``; such a build goes to ``out`` instead of the default
library path.  ``build_phases`` (``--phases``) builds the diagnostic variant
with the wave kernels' phase stamps compiled in,
``libllcoll_phases.so``, which ``timeline.py`` loads.
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libllcoll.so")
PHASES_LIB = os.path.join(HERE, "libllcoll_phases.so")
ARCH = os.environ.get("LLCOLL_ARCH", "gfx950")
RANKS = range(2, 9)

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # no packed fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # IEEE subnormals and no fused operations: the sums must be exact binary32 adds
    "-fno-gpu-flush-denormals-to-zero",
    "-ffp-contract=off",
    "-Wall",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "packed-fp32-ops"  # the host pass does not know the device feature; harmless
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    return res.returncode, msgs


def build(verbose: bool = False, extra_defines=(), out: str | None = None, jobs: int | None = None) -> str:
    target = out or LIB
    defs = [f"-D{d}" for d in extra_defines]
    with tempfile.TemporaryDirectory(prefix="llcoll_build_") as tmp:
        units = [([os.path.join(CSRC, "llcoll.hip")], os.path.join(tmp, "llcoll.o"))]
        for p in RANKS:
            units.append(([f"-DLL_INST_P={p}", os.path.join(CSRC, "ll_inst.hip")], os.path.join(tmp, f"ll_inst_p{p}.o")))
        cmds = [[hipcc(), *HIPCC_FLAGS, *defs, "-c", *src, "-o", obj] for src, obj in units]
        workers = jobs or max(1, min(len(cmds), os.cpu_count() or 1, 16))
        with ThreadPoolExecutor(max_workers=workers) as pool:
            results = list(pool.map(_run, cmds))
        for (rc, msgs), cmd in zip(results, cmds):
            if rc != 0:
                raise RuntimeError(f"hipcc failed ({rc}): {' '.join(cmd)}\n{msgs}")
            if verbose and msgs.strip():
                print(msgs, file=sys.stderr)
        tmp_lib = target + ".tmp"
        rc, msgs = _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp_lib,
                         *[obj for _, obj in units]])
        if rc != 0:
            raise RuntimeError(f"link failed ({rc}):\n{msgs}")
    os.replace(tmp_lib, target)
    return target


def build_phases(verbose: bool = False) -> str:
    return build(verbose, extra_defines=("LLCOLL_WAVE_PHASES=1",), out=PHASES_LIB)


if __name__ == "__main__":
    if "--phases" in sys.argv[1:]:
        print(build_phases(verbose=True))
    else:
        print(build(verbose=True))
