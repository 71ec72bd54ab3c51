"""Build libmkv.so (HIP kernels for gfx950 + the C-ABI host library) in place.

    python -m paper_2609_07966_amd.build            # or build() from Python

The library is written next to this file so that it travels with the source tree.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libmkv.so")

SOURCES = ["mkv_api.cpp", "calib.cpp", "select.cpp", "k_attn.hip", "k_append.hip", "k_select.hip", "k_probe.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"


def flags():
    return [
        "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
        # no packed fp32 instructions in device code; no implicit fused multiply-add (the
        # quantizer and approximate-score steps are specified in separately rounded float32)
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # matrix-core accumulators in ordinary VGPRs: the attention loop rescales them with VALU
        # ops, which cannot read the accumulation registers
        "-mllvm", "-amdgpu-mfma-vgpr-form",
        "-ffp-contract=off", "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
        "-I", os.path.join(ROOT, "include"), "-I", CSRC,
    ]


def build(verbose=False, jobs=None):
    """Compile every source to an object in parallel, then link libmkv.so."""
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    procs = []
    objs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src + ".o")
        objs.append(obj)
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = [HIPCC] + [f for f in flags() if f != "-shared"] + ["-c"] + lang + [os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    failed = []
    for src, p in procs:
        out = p.communicate()[0].decode(errors="replace")
        out = "\n".join(l for l in out.splitlines() if "packed-fp32-ops" not in l and "is not a recognized feature" not in l)
        if p.returncode != 0:
            failed.append((src, out))
        elif verbose and out.strip():
            print(out)
    if failed:
        for src, out in failed:
            sys.stderr.write(f"---- {src} ----\n{out}\n")
        raise RuntimeError("libmkv build failed: " + ", ".join(s for s, _ in failed))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", "-o", tmp] + objs
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
