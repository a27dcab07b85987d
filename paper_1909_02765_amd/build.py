"""Build libilpm.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

    python paper_1909_02765_amd/build.py            # build in-tree
    python paper_1909_02765_amd/build.py --isa DIR  # also keep the gfx950 assembly in DIR

(Run it as a script: importing the package loads the library it builds.)
"""
from __future__ import annotations

import argparse
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "libilpm.so")

ARCH = "gfx950"
# Packed fp32 VALU instructions stay disabled: the compiler forms them on its
# own from scalar float code, and they are not needed here (the dense path
# uses the fp32 matrix cores).
# MFMA accumulators in ordinary VGPRs (the register file is unified on gfx950):
# measured faster than the AGPR form on these kernels (1-8% per variant), which
# made the compiler shuttle accumulators between the two register classes.
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]
FLAGS = ["-O3", "-std=c++17", f"--offload-arch={ARCH}", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"] + VGPR_FORM + [
         "-Wall", "-Wno-unused-function", "-Wno-unused-command-line-argument"]
# Sources built in the compiler's default accumulator form instead: one
# instantiation of a variant there computed wrong values in the VGPR form
# (found by the bit-exact epilogue tests; right in the default form).
DEFAULT_FORM_SOURCES = {"conv_igemm_v8.hip"}


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def hipcc() -> str:
    p = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    return p


def _compile(src: str, obj: str, extra=(), cwd=None, verbose=False):
    flags = [f for f in FLAGS if f != "-shared"]
    if os.path.basename(src) in DEFAULT_FORM_SOURCES:
        flags = [f for f in flags if f not in VGPR_FORM]
    cmd = [hipcc()] + flags + ["-I", INCLUDE, "-I", CSRC] + list(extra)
    cmd += ["-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True, cwd=cwd)
    return obj


def build(output: str = LIBRARY, isa_dir: str | None = None, verbose: bool = False, jobs: int = 0) -> str:
    """Compile every csrc/*.hip to an object (in parallel: the matrix-core
    variants are spread over several files for this), then link the shared
    library.  With isa_dir, the intermediate files (gfx950 assembly) are kept
    there."""
    import tempfile
    from concurrent.futures import ThreadPoolExecutor
    srcs = sources()
    jobs = jobs or min(len(srcs), os.cpu_count() or 1, 16)
    with tempfile.TemporaryDirectory(prefix="ilpm_build_") as tmpdir:
        objdir = isa_dir or tmpdir
        if isa_dir:
            os.makedirs(isa_dir, exist_ok=True)
        extra = ["-save-temps=obj"] if isa_dir else []
        objs = [os.path.join(objdir, os.path.basename(sp) + ".o") for sp in srcs]
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            futs = [ex.submit(_compile, sp, ob, extra, objdir if isa_dir else None, verbose)
                    for sp, ob in zip(srcs, objs)]
            for f in futs:
                f.result()
        tmp = output + ".tmp"
        cmd = [hipcc()] + FLAGS + objs + ["-o", tmp]
        if verbose:
            print(" ".join(cmd), file=sys.stderr)
        subprocess.run(cmd, check=True)
    os.replace(tmp, output)
    return output


PEAKS_SOURCE = os.path.join(ROOT, "bench_peaks.hip")
PEAKS_LIBRARY = os.path.join(ROOT, "bench_peaks.so")


def build_peaks(output: str = PEAKS_LIBRARY) -> str:
    """The peak microbenchmarks used by bench.py --peaks."""
    tmp = output + ".tmp"
    subprocess.run([hipcc()] + FLAGS + [PEAKS_SOURCE, "-o", tmp], check=True)
    os.replace(tmp, output)
    return output


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--isa", default=None, help="keep intermediate files (gfx950 assembly) here")
    ap.add_argument("-v", action="store_true")
    args = ap.parse_args()
    print(build(isa_dir=args.isa, verbose=args.v))
    print(build_peaks())


if __name__ == "__main__":
    main()
