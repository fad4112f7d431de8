"""Build libmtn.so (host library + gfx950 kernels) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmtn.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 VALU ops stay off: ordinary float code only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
    "-Wall", "-Wno-unused-function", "-Wno-unused-result",
]

SOURCES = ["mtn_host.cpp", "mtn_admission.cpp", "mtn_kernels.hip", "mtn_mfma.hip"]

# Per-source code generation.  The matrix-core decode takes its MFMA
# accumulators in ordinary VGPRs: in the AGPR form the compiler copied the 32
# output accumulators out of and back into AGPRs around every block's rescale
# test (about 100 of its 250 vector instructions per block; measured 1.3 %
# faster fp8 and 0.4 % faster bf16 launches without them).
EXTRA = {"mtn_mfma.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def compile_flags(src: str) -> list:
    """Every option `src` is compiled with (part of the key of the committed
    counter summaries, since the flags shape the kernels as the code does)."""
    return [*COMMON, *EXTRA.get(src, [])]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd[:3])} ...")
    # the host pass does not know the packed-fp32 feature flag; drop that noise
    noise = "is not a recognized feature for this target"
    rest = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if rest.strip() and verbose:
        print(rest)


def build(verbose: bool = False, out: str = LIB, defines=()) -> str:
    """Compile every source for gfx950 and link libmtn.so next to this file
    (or at ``out``, with extra ``-D`` ``defines`` for tuning variants)."""
    objs = []
    tag = "_".join("".join(ch for ch in d if ch.isalnum()) for d in defines)
    bdir = os.path.join(ROOT, "_build", tag) if tag else os.path.join(ROOT, "_build")
    os.makedirs(bdir, exist_ok=True)
    for src in SOURCES:
        obj = os.path.join(bdir, src + ".o")
        _run([HIPCC, *compile_flags(src), *[f"-D{d}" for d in defines], "-c",
              os.path.join(CSRC, src), "-o", obj], verbose)
        objs.append(obj)
    tmp = out + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, out)
    return out


SANITIZED = os.path.join(ROOT, "_build", "sanitize", "libmtn_host_sanitized.so")


def build_host_sanitized(verbose: bool = False, out: str = SANITIZED) -> str:
    """The host library alone (planner, tables, admission) built by g++ with
    AddressSanitizer and UndefinedBehaviorSanitizer, the gfx950 launch
    interface replaced by host stand-ins (mtn_host_stub.cpp).  Only host-only
    pools work with it; load it with the sanitizer runtime preloaded."""
    os.makedirs(os.path.dirname(out), exist_ok=True)
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{INCLUDE}", f"-I{CSRC}",
           os.path.join(CSRC, "mtn_host.cpp"), os.path.join(CSRC, "mtn_admission.cpp"),
           os.path.join(CSRC, "mtn_host_stub.cpp"), "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,/opt/rocm/lib", "-o", out + ".tmp"]
    _run(cmd, verbose)
    os.replace(out + ".tmp", out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
