"""Build libndvm.so in-tree for gfx950 with hipcc.

Kernels and host code are compiled with -ffp-contract=off (no implicit fused
multiply-add: every +, -, *, / is one IEEE operation, matching the oracle)
and with packed-fp32 instructions disabled.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libndvm.so")
# host emulator of device programs: a scheduler-checking tool loaded only by the CPU tests
EMU_OUT = os.path.join(HERE, "libndvm_emu.so")
BUILD = os.path.join(HERE, "_build")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["frontend.cpp", "tape.cpp", "sched.cpp", "abi.cpp", "kernels.hip", "optim.hip", "walk_host.cpp", "walk.hip"]
EMU_SOURCES = ["frontend.cpp", "tape.cpp", "sched.cpp", "emu.cpp"]
COMMON = ["-O3", "-fPIC", "-std=c++17", "-ffp-contract=off", "-fno-fast-math", "-Wall",
          "-Wno-unused-function"]
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
# the replay kernel's options
REPLAY = [
    # the interpreter's dispatch branches are wave-uniform: leave such
    # regions unstructured instead of routing every handler exit through a
    # chain of flow blocks
    "-mllvm", "-structurizecfg-skip-uniform-regions=true",
    # keep every handler's final register store in the handler: sunk into a
    # shared block it would wait there for the memory traffic of every other
    # handler (the program prefetch included)
    "-mllvm", "-sink-common-insts=false", "-mllvm", "-enable-tail-merge=false"]
# sources built with the replay kernel's options (the device walker is not:
# with its loops the first option makes the code generator fail)
REPLAY_OPTIONS_FOR = {"frontend.cpp", "tape.cpp", "sched.cpp", "abi.cpp", "kernels.hip", "optim.hip", "emu.cpp"}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    extra = REPLAY if src in REPLAY_OPTIONS_FOR else []
    cmd = [HIPCC] + COMMON + DEVICE + extra + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stderr or "").splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def _link(objs, out):
    tmp = out + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}"] + objs + ["-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(set(SOURCES) | set(EMU_SOURCES))
    with ThreadPoolExecutor(max_workers=len(srcs)) as ex:
        objs = dict(zip(srcs, ex.map(_compile, srcs)))
    _link([objs[s] for s in SOURCES], OUT)
    _link([objs[s] for s in EMU_SOURCES], EMU_OUT)
    if verbose:
        print("built", OUT, "and", EMU_OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
