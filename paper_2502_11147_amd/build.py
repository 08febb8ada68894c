"""Compiles the HIP sources of the decode path into ``libraas.so`` (gfx950)."""
from __future__ import annotations

import hashlib
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(HERE, "libraas.so")
SOURCES = [os.path.join(CSRC, "raas_kernels.hip"), os.path.join(CSRC, "raas_runtime.hip")]
# the streaming probe (measurement only) is a library of its own
PROBE_SOURCES = [os.path.join(CSRC, "raas_probe.hip")]
PROBE_LIB_PATH = os.path.join(HERE, "libraas_probe.so")
ARCH = "gfx950"


def hipcc_command(out: str, sources=None) -> list[str]:
    return [
        "hipcc", "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
        # packed fp32 vector instructions stay off on this target
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-I", INCLUDE, "-I", CSRC, *(SOURCES if sources is None else sources), "-o", out,
    ]


def _code_text(src: str) -> str:
    """C++ source without its comments and with whitespace runs collapsed
    (the kernels' sources hold no comment markers inside literals)."""
    out, i, n = [], 0, len(src)
    while i < n:
        if src.startswith("//", i):
            j = src.find("\n", i)
            i = n if j < 0 else j
        elif src.startswith("/*", i):
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(src[i])
            i += 1
    return " ".join("".join(out).split())


def kernel_digest() -> str:
    """sha256 over the kernel sources' code (comments and layout left out)
    and the compile flags: identifies the kernels that a stored
    hardware-counter measurement was taken on."""
    h = hashlib.sha256()
    for p in (os.path.join(CSRC, "raas_kernels.hip"), os.path.join(CSRC, "raas_internal.h")):
        with open(p, encoding="utf-8") as f:
            h.update(_code_text(f.read()).encode())
    h.update(" ".join(a for a in hipcc_command("lib") if not os.path.isabs(a) and a not in ("-I", "-o", "lib")).encode())
    return h.hexdigest()


def _compile(out: str, sources, verbose: bool):
    tmp = out + ".tmp%d" % os.getpid()
    cmd = hipcc_command(tmp, sources)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)
    if verbose:
        print(" ".join(cmd))
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    """Builds libraas.so (the decode path) and libraas_probe.so (the
    streaming probe of the measurements)."""
    _compile(LIB_PATH, SOURCES, verbose)
    _compile(PROBE_LIB_PATH, PROBE_SOURCES, verbose)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
