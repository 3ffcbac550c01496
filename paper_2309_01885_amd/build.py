"""Builds libqe.so (the HIP library behind include/qe.h) and libqe_peak.so
(peak-check probes) for gfx950, in-tree."""
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libqe.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-result",
    # keep the compiler from forming packed fp32 instructions (v_pk_*_f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


PEAK_SRC = os.path.join(HERE, "peak", "peak.hip")
PEAK_LIB = os.path.join(HERE, "libqe_peak.so")


def _hipcc(srcs, out, verbose):
    tmp = out + ".tmp"
    cmd = [HIPCC] + FLAGS + srcs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stderr or "").splitlines() if noise not in l)
    if r.returncode != 0:
        sys.stderr.write(err + "\n")
        raise RuntimeError(f"hipcc failed building {os.path.basename(out)}")
    if verbose and err.strip():
        sys.stderr.write(err + "\n")
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    """libqe.so (the C ABI of include/qe.h) and libqe_peak.so (peak checks)."""
    _hipcc([PEAK_SRC], PEAK_LIB, verbose)
    return _hipcc(sources(), LIB, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
