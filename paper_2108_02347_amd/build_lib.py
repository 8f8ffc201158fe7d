"""Builds libfmm_attn.so in-tree with hipcc for gfx950.

Usage: python -m paper_2108_02347_amd.build_lib   (or call build())
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libfmm_attn.so")
SOURCES = ["fmm_kernels.hip", "fmm_wide.hip", "fmm_bwd.hip", "fmm_pair.hip", "fmm_causal.hip",
           "fmm_noalloc.hip", "fmm_layer.hip", "fmm_fastweight.hip", "fmm_api.cpp"]
# translation units compiled a second time with other options: (source, object
# name, extra flags, whether MFMA results are forced into vector registers)
VARIANTS = [
    # the backward's fp32 d = 128 passes: one workgroup per CU, with the
    # accumulation registers beside the vector registers
    ("fmm_bwd.hip", "fmm_bwd_f32_d128", ["-DFMM_BWD_F32_D128"], False),
]
HEADERS = ["fmm_device.h", "fmm_launch.h", "fmm_oct.h", "fmm_apply.h", "fmm_fw.h"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; the HIP library cannot be built")


def _flags(vgpr_form: bool = True):
    f = [
        "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
        # keep the compiler from forming packed fp32 instructions
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    ]
    if vgpr_form:
        # keep MFMA accumulators in ordinary VGPRs: the kernels scale and
        # blend them with VALU code, which would otherwise copy them out of
        # and back into AGPRs
        f += ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]
    return f + ["-Wno-unused-result", "-I", os.path.join(ROOT, "include")]


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 into LIB (always recompiles).  The
    translation units are compiled in parallel, then linked."""
    cc = hipcc()
    tmpdir = tempfile.mkdtemp(prefix="fmm_build_")
    try:
        objs, procs = [], []
        units = [(src, src, [], True) for src in SOURCES] + VARIANTS
        for src, name, extra, vgpr_form in units:
            obj = os.path.join(tmpdir, name + ".o")
            cmd = [cc] + _flags(vgpr_form) + extra + ["-c", os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            procs.append((name, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                 stderr=subprocess.STDOUT, text=True)))
            objs.append(obj)
        failed = []
        for src, pr in procs:
            out, _ = pr.communicate()
            if pr.returncode != 0:
                sys.stderr.write(out)
                failed.append(src)
            elif verbose and out.strip():
                sys.stderr.write(out)
        if failed:
            raise RuntimeError(f"hipcc failed on {', '.join(failed)}")
        # rocBLAS serves the attention layer's projections
        cmd = ([cc, "--offload-arch=gfx950", "-shared", "-fPIC"] + objs +
               ["-L/opt/rocm/lib", "-lrocblas", "-Wl,-rpath,/opt/rocm/lib", "-o", LIB + ".tmp"])
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError(f"hipcc link failed with status {res.returncode}")
        os.replace(LIB + ".tmp", LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
