"""Build step of the SAEF HIP library: hipcc for gfx950 into libsaef.so (in-tree).

Flags: no FMA contraction (every a*b+c in the kernels is an explicit fma),
no fast-math, fp32 denormals kept, packed-fp32 instructions disabled.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = [os.path.join(HERE, "csrc", f) for f in ("saef_kernels.hip", "saef_topk.hip",
                                                          "saef_api.hip")]
LIB = os.path.join(HERE, "libsaef.so")
# the same library with 4096-element work tiles: the tile-size determinism
# test runs the sign path with both builds and compares the bytes
TILE_VARIANT_ELEMS = 4096
LIB_TILE_VARIANT = os.path.join(HERE, f"libsaef_tile{TILE_VARIANT_ELEMS}.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fno-fast-math", "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wextra", "-Werror",
]


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    path = os.path.join(rocm, "bin", "hipcc")
    return path if os.path.exists(path) else "hipcc"


def build(out: str = LIB, verbose: bool = False, defines=()) -> str:
    """Compile the library to `out`; `defines` are extra -D options (tuning
    variants, e.g. SAEF_TILE_ELEMS=2048)."""
    cmd = [hipcc(), *HIPCC_FLAGS, *[f"-D{d}" for d in defines],
           "-I", os.path.join(ROOT, "include"), "-o", out + ".tmp", *SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # the host pass does not know the packed-fp32 feature and says so; harmless
    noise = [ln for ln in res.stderr.splitlines() if "packed-fp32-ops" not in ln
             and "warning generated" not in ln and ln.strip()]
    if res.returncode != 0:
        sys.stderr.write(res.stderr)
        raise RuntimeError(f"hipcc failed ({res.returncode})")
    if verbose and noise:
        sys.stderr.write("\n".join(noise) + "\n")
    os.replace(out + ".tmp", out)
    return out


CLIENT_SRC = os.path.join(ROOT, "tests", "c", "abi_client.cpp")
CLIENT = os.path.join(ROOT, "tests", "c", "abi_client")


def build_client(out: str = CLIENT, lib: str = LIB) -> str:
    """Compile the C/C++ client of the C ABI (tests/c/abi_client.cpp) against
    the built library; it finds the library through a relative run path."""
    libdir = os.path.dirname(lib)
    rel = os.path.relpath(libdir, os.path.dirname(out))
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-O2", "-std=c++17", "-Wall", "-Werror",
           "-I", os.path.join(ROOT, "include"), CLIENT_SRC, "-L", libdir,
           f"-l:{os.path.basename(lib)}", f"-Wl,-rpath,$ORIGIN/{rel}", "-o", out + ".tmp"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stderr)
        raise RuntimeError(f"hipcc failed ({res.returncode})")
    os.replace(out + ".tmp", out)
    return out


def build_tile_variant(verbose: bool = False) -> str:
    """The library with SAEF_TILE_ELEMS = TILE_VARIANT_ELEMS (Top-K plans are
    refused by that build; the sign path is complete)."""
    return build(out=LIB_TILE_VARIANT, verbose=verbose,
                 defines=(f"SAEF_TILE_ELEMS={TILE_VARIANT_ELEMS}",))


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_tile_variant())
    print(build_client())
