"""Build steps for the native libraries (run on the CPU; hipcc cross-compiles gfx950).

* ``libparason.so``      -- the hot path: HIP kernels + C-ABI (``csrc/parason.hip``,
  ``csrc/pg.hip``, ``csrc/decode.hip``, ``csrc/fork.hip``)
* ``libparason_synth.so``-- device side of the synthetic generator (``synth/synth.hip``)
* ``libparason_synth_host.so`` -- host mirror of the generator (g++)

Everything is built in-tree, next to its sources, so the libraries travel with
the repository snapshot.
"""
from __future__ import annotations

import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
INCLUDE = os.path.join(ROOT, "include")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Device code: no packed-fp32 instructions, no FMA contraction (the reward is
# evaluated in a fixed order), -O3.
HIP_FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]

LIBS = {
    "parason": dict(
        out=os.path.join(PKG, "libparason.so"),
        srcs=[os.path.join(PKG, "csrc", f) for f in ("parason.hip", "pg.hip", "decode.hip", "fork.hip")],
        deps=[os.path.join(PKG, "csrc", f) for f in ("abi_common.h", "device_common.h", "parason_kernels.h",
                                                       "pg_kernels.h", "decode_kernels.h", "fork_kernels.h")]
        + [os.path.join(INCLUDE, "parason.h")],
        kind="hip",
    ),
    "synth": dict(
        out=os.path.join(PKG, "synth", "libparason_synth.so"),
        srcs=[os.path.join(PKG, "synth", "synth.hip")],
        deps=[os.path.join(PKG, "synth", "synth_core.h")],
        kind="hip",
    ),
    "synth_host": dict(
        out=os.path.join(PKG, "synth", "libparason_synth_host.so"),
        srcs=[os.path.join(PKG, "synth", "synth_host.cpp")],
        deps=[os.path.join(PKG, "synth", "synth_core.h")],
        kind="host",
    ),
}


def _cmd(spec, out):
    if spec["kind"] == "hip":
        return [HIPCC] + HIP_FLAGS + ["-I", INCLUDE, "-o", out] + spec["srcs"]
    return [
        "g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-ffp-contract=off",
        "-D__host__=", "-D__device__=", "-Wall", "-o", out,
    ] + spec["srcs"]


def stale(name: str) -> bool:
    spec = LIBS[name]
    if not os.path.exists(spec["out"]):
        return True
    t = os.path.getmtime(spec["out"])
    return any(os.path.exists(p) and os.path.getmtime(p) > t for p in spec["srcs"] + spec["deps"])


def build_one(name: str, verbose: bool = False) -> str:
    spec = LIBS[name]
    tmp = spec["out"] + ".tmp%d" % os.getpid()
    cmd = _cmd(spec, tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, spec["out"])
    return spec["out"]


def build_all(verbose: bool = False, only_stale: bool = False) -> None:
    for name in LIBS:
        if only_stale and not stale(name):
            continue
        build_one(name, verbose=verbose)


if __name__ == "__main__":
    build_all(verbose=True)
