"""Build libsparsp.so (the HIP kernels and the C ABI) in-tree for gfx950.

Usage: python -m paper_2609_32197_amd.build [--jobs N] [--verbose]

Each .hip file under csrc/ is compiled with hipcc for gfx950 only; each .cpp
file there (the C ABI layer and the pure host planning code, which use only
the HIP runtime API) with the host C++ compiler. Both are linked into
paper_2609_32197_amd/libsparsp.so next to this file. Packed fp32 VALU
instructions are disabled for device code (they are not used by these kernels
and some of their forms are avoided on purpose).

The benchmark's measurement helper, probe/mfma_probe.hip, is built into its
own library, probe/libmfma_probe.so: it is not part of libsparsp.
"""

from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libsparsp.so")
PROBE_SRC = os.path.join(HERE, "probe", "mfma_probe.hip")
PROBE_LIB = os.path.join(HERE, "probe", "libmfma_probe.so")
ARCH = "gfx950"
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

# Host-only C++ (no device code): the HIP runtime API headers, AMD platform.
HOST_COMMON = [
    "-O2",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wextra",
    "-Wno-unused-parameter",
    "-D__HIP_PLATFORM_AMD__",
    f"-I{os.path.join(ROCM, 'include')}",
    f"-I{os.path.join(ROOT, 'include')}",
]

COMMON = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{os.path.join(ROOT, 'include')}",
]


# Extra flags per source. The bf16 attention kernel never sees NaN (inputs are
# finite, masked keys are -inf), so fmaxf needs no NaN quieting; infinities are
# still honoured.
PER_FILE = {"attn_bf16.hip": ["-fno-honor-nans"]}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


def host_cxx() -> str:
    for cand in (os.environ.get("CXX"), shutil.which("g++"), shutil.which("c++")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("no host C++ compiler found (set CXX)")


def sources() -> list:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def host_sources() -> list:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".cpp"))


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # hipcc's host pass warns that it does not know the packed-fp32 feature: harmless.
    noise = "not a recognized feature for this target"
    msg = "\n".join(x for x in (r.stdout + r.stderr).splitlines() if noise not in x
                    and "(ignoring feature)" not in x)
    if msg.strip() and verbose:
        print(msg)
    return r


def build(jobs: int = 8, verbose: bool = False) -> str:
    """Compile every source and link the shared library; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    srcs = sources()
    objs = [os.path.join(BUILD, os.path.basename(s)[:-4] + ".o") for s in srcs]
    cmds = [[cc, *COMMON, *PER_FILE.get(os.path.basename(s), []), "-c", s, "-o", o]
            for s, o in zip(srcs, objs)]
    hsrcs = host_sources()
    hobjs = [os.path.join(BUILD, os.path.basename(s)[:-4] + ".host.o") for s in hsrcs]
    cmds += [[host_cxx(), *HOST_COMMON, "-c", s, "-o", o] for s, o in zip(hsrcs, hobjs)]
    probe_tmp = PROBE_LIB + ".tmp"
    cmds.append([cc, *COMMON, "-shared", PROBE_SRC, "-o", probe_tmp])
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    os.replace(probe_tmp, PROBE_LIB)
    tmp = LIB + ".tmp"
    _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, *hobjs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--jobs", type=int, default=min(8, os.cpu_count() or 1))
    ap.add_argument("--verbose", action="store_true")
    a = ap.parse_args(argv)
    print(build(a.jobs, a.verbose))
    return 0


if __name__ == "__main__":
    sys.exit(main())
