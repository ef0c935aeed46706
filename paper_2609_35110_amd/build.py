"""Build libsol.so (HIP kernels for gfx950 + the C ABI) in-tree with hipcc."""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libsol.so")
# debug build: LDS arrays that hold values are filled with NaN at kernel entry
POISON_LIB = os.path.join(PKG, "libsol_poison.so")
SOURCES = ["sol_kernels.hip", "sol_sparse.hip", "sol_records.hip", "sol_probe.hip", "sol_noalloc.hip",
           "sol_api.cpp"]
ARCH = "gfx950"

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared",
    "--offload-arch=" + ARCH,
    # every multiply/add in the kernels is written out; no silent contraction
    "-ffp-contract=off",
    # no NaN arises in the kernels' own arithmetic (masking uses -inf): lets
    # max reductions compile to v_max3 without NaN canonicalisation
    "-fno-honor-nans",
    # no packed fp32 VALU instructions (v_pk_*_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # loop heads on a 64-byte boundary: a one-wave-per-SIMD loop refetches
    # its first instructions on every back edge (measured 1.5 % on the
    # attention kernel between the good and bad offsets)
    "-falign-loops=64",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    return path


def build(verbose: bool = False, poison: bool = False) -> str:
    """Compile every HIP/C++ source into paper_2609_35110_amd/libsol.so (always
    rebuilds).  poison: the LDS-poison debug build, libsol_poison.so (the same
    sources with -DSOL_LDS_POISON)."""
    out = POISON_LIB if poison else LIB
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    tmp = out + ".tmp%d" % os.getpid()
    defs = ["-DSOL_LDS_POISON"] if poison else []
    cmd = [hipcc()] + HIPCC_FLAGS + defs + ["-I", INCLUDE, "-I", CSRC, "-x", "hip"] + srcs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the packed-fp32 target feature; that warning is harmless
    noise = ("packed-fp32-ops", "not a recognized feature", "(ignoring feature)")
    msgs = [ln for ln in (res.stdout + res.stderr).splitlines() if ln.strip() and not any(n in ln for n in noise)]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s" % (res.returncode, "\n".join(msgs)))
    if msgs and verbose:
        print("\n".join(msgs))
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, poison="--poison" in sys.argv))
