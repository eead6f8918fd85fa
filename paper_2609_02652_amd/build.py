"""Build libleech.so (HIP for gfx950 + host C++) in place, next to this file.

    python paper_2609_02652_amd/build.py

Every HIP source is compiled for gfx950 with packed-FP32 instructions
disabled (-Xclang -target-feature -Xclang -packed-fp32-ops); the host pass of
hipcc warns that it does not know that feature, which is harmless.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libleech.so")
SOURCES = [os.path.join(CSRC, "host.cpp"), os.path.join(CSRC, "kernels.hip"),
           os.path.join(CSRC, "rotate.hip"), os.path.join(CSRC, "transcode.hip")]
ARCH = os.environ.get("LEECH_OFFLOAD_ARCH", "gfx950")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    return "hipcc"


def command(out: str = LIB) -> list:
    return [hipcc(), "-std=c++17", "-O3", "-fPIC", "-shared", f"--offload-arch={ARCH}",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-Wno-unused-parameter",
            f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", *SOURCES, "-o", out, "-lpthread"]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = command(tmp)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in proc.stderr.splitlines() if noise not in l)
    if proc.returncode != 0:
        raise RuntimeError("libleech build failed:\n" + " ".join(cmd) + "\n" + err)
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
