"""Build the HIP library ``libqlin.so`` in-tree for gfx950 with hipcc.

``python -m paper_2607_04244_amd.build`` (or ``__graft_entry__.build()``)
compiles every source under ``csrc/`` on each call.  It also links
``libqlin_asan.so``: the same device code, with the host-only C-ABI sources
(argument checks, planner, handle management) compiled by g++ with
AddressSanitizer and UndefinedBehaviorSanitizer, for the CPU tests of the
ABI (the sanitizer runtimes are preloaded into the Python that loads it).
"""

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libqlin.so")
# (source, extra flags).  tiled.hip and attn.hip keep matrix-core results in
# VGPRs: their products feed vector instructions directly (dequantization,
# softmax rescaling), which would otherwise go through AGPR copies.
SOURCES = [("kernels.hip", []), ("tiled.hip", ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]), ("attn.hip", ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]),
           ("qlin.cpp", []), ("attn_abi.cpp", [])]
HOST_SOURCES = ("qlin.cpp", "attn_abi.cpp")       # no device code: plain C++ against the HIP headers
LIB_ASAN = os.path.join(HERE, "libqlin_asan.so")
SANITIZE = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
ARCH = "gfx950"

# Packed-fp32 vector instructions are switched off in the device pass; the
# host pass warns that it does not know the feature, which is harmless.
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]
NOISE = "is not a recognized feature for this target"


def _errs(r):
    return "\n".join(l for l in (r.stderr or "").splitlines() if NOISE not in l)


def build(verbose=False, extra_flags=()):
    """Compile every source to an object (in parallel), then link the library."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    inc = ["-I", os.path.join(HERE, "..", "include")]
    objs, procs = [], []
    for src, flags in SOURCES:
        obj = os.path.join(CSRC, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc, *HIP_FLAGS, *flags, *extra_flags, *inc, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True)))
        objs.append(obj)
    failed = []
    for src, p in procs:
        out, err = p.communicate()
        r = subprocess.CompletedProcess(p.args, p.returncode, out, err)
        if r.returncode != 0:
            failed.append(f"{src}:\n{_errs(r)}")
        elif verbose and _errs(r).strip():
            print(_errs(r), file=sys.stderr)
    if failed:
        raise RuntimeError("hipcc failed:\n" + "\n".join(failed))
    # the host sources again, instrumented, for the sanitizer library
    cxx = os.environ.get("CXX_HOST", "g++")
    asan_objs = []
    for src in HOST_SOURCES:
        obj = os.path.join(CSRC, os.path.splitext(src)[0] + ".asan.o")
        cmd = [cxx, "-O1", "-g", "-std=c++17", "-fPIC", *SANITIZE, "-D__HIP_PLATFORM_AMD__",
               "-I", "/opt/rocm/include", *inc, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"{cxx} failed on {src}:\n{r.stderr}")
        asan_objs.append(obj)
    device_objs = [o for (src, _), o in zip(SOURCES, objs) if src not in HOST_SOURCES]
    for out, parts in ((LIB, objs), (LIB_ASAN, device_objs + asan_objs)):
        tmp = out + ".tmp"
        cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *parts, "-o", tmp]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed ({r.returncode}):\n{_errs(r)}")
        os.replace(tmp, out)
    for o in objs + asan_objs:
        os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
