"""Compile the HIP sources in csrc/ into libqf.so (gfx950) next to this file.

Flags: -ffp-contract=off keeps every FP32 step of the quantizers a single IEEE operation
(results are bit-exact across implementations); packed FP32 ops are disabled for all device
code.  The C ABI is declared in include/qf.h at the repository root.
"""
import glob
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libqf.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = ["-O3", "-std=c++17", "-fPIC", "-shared", "--offload-arch=" + ARCH,
         "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-fvisibility=hidden", "-Wall"]


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC] + FLAGS + ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"),
                             "-o", tmp] + sources()
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + err)
    if verbose and err.strip():
        print(err)
    check_stubs(tmp)
    os.replace(tmp, LIB)
    return LIB


def check_stubs(path: str) -> None:
    """Fail if a kernel's host launch stub is left undefined (the library would load-fail)."""
    r = subprocess.run(["nm", "--undefined-only", path], capture_output=True, text=True)
    if r.returncode != 0:
        return
    bad = [l.split()[-1] for l in r.stdout.splitlines() if "__device_stub" in l]
    if bad:
        raise RuntimeError("undefined kernel launch stubs in %s: %s" % (path, bad))


if __name__ == "__main__":
    print(build(verbose=True))
