"""Build libsfl.so (HIP kernels for gfx950 + the C ABI) in-tree with hipcc.

Every source under csrc/ is compiled to an object file in parallel, then linked
into `libsfl.so` next to this file. The build always recompiles (it is the
"does it build" check); `python -m paper_2603_23198_amd.build` runs it.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsfl.so")
ARCH = "gfx950"  # the kernels use CDNA4 instructions (MFMA 16x16x32 bf16, ds_read_b64_tr_b16)

FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # keep the compiler from emitting packed fp32 arithmetic (v_pk_* f32)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-munsafe-fp-atomics",
    # the GEMM epilogues index their accumulator arrays from fully unrolled loops; let the
    # unroller expand them however large, so the arrays stay in registers
    "-mllvm", "-pragma-unroll-threshold=1000000",
    "-Wno-unused-result",
]


def hipcc():
    for c in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _compile(src, obj, extra=()):
    cmd = [hipcc(), *FLAGS, *extra, "-x", "hip", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in (r.stderr or "").splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {os.path.basename(src)}:\n{errs}")
    return errs


def build(verbose=False, jobs=None, extra_flags=(), out=None, csrc=None) -> str:
    """Compile and link; `extra_flags` go to every hipcc line, `out` overrides the library
    path and `csrc` the source directory."""
    lib = out or LIB
    src_dir = csrc or CSRC
    srcs = sorted(glob.glob(os.path.join(src_dir, "*.hip")) + glob.glob(os.path.join(src_dir, "*.cpp")))
    jobs = jobs or min(len(srcs), max(1, (os.cpu_count() or 4)), 16)
    with tempfile.TemporaryDirectory(prefix="sfl_build_") as tmp:
        objs = [os.path.join(tmp, os.path.basename(s) + ".o") for s in srcs]
        with cf.ThreadPoolExecutor(jobs) as ex:
            for src, msg in zip(srcs, ex.map(lambda a, o: _compile(a, o, extra_flags), srcs, objs)):
                if verbose and msg.strip():
                    print(f"[{os.path.basename(src)}]\n{msg}", file=sys.stderr)
        tmp_lib = lib + ".tmp"
        cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp_lib]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed:\n{r.stderr}")
        os.replace(tmp_lib, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True))
