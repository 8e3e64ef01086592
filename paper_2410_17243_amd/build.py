"""Build libinfcl.so (the HIP kernels and the C ABI) in-tree for gfx950.

    python -m paper_2410_17243_amd.build [--verbose]

Every call recompiles.  Each HIP source is compiled to an object in parallel,
then the objects are linked into ``paper_2410_17243_amd/libinfcl.so``.  The
device assembly of every source (kept from the same compilation) is checked
for the wait states of its inline-assembly MFMA and DMA instructions
(``waitstates.py``); a violation fails the build.
"""

from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libinfcl.so")
SOURCES = ["api.hip", "fwd.hip", "fwd2.hip", "bwd.hip", "bwd_wide.hip", "ablation.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    # packed fp32 VALU forms are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libinfcl.so)")


def device_asm_path(workdir: str, src: str) -> str:
    """Device assembly that -save-temps leaves for `src` in `workdir`."""
    return os.path.join(workdir, src[: -len(".hip")] + "-hip-amdgcn-amd-amdhsa-gfx950.s")


def build(verbose: bool = False, resource_usage: bool = False, defines=(), out: str = LIB,
          check_waits: bool = True) -> str:
    """Compile and link; `defines` are extra -D options (build-time tuning knobs)."""
    from . import waitstates

    cc = hipcc()
    tmp = tempfile.mkdtemp(prefix="infcl_build_")
    try:
        def compile_one(src):
            work = os.path.join(tmp, src)
            os.makedirs(work)
            obj = os.path.join(tmp, src + ".o")
            cmd = [cc, *HIPCC_FLAGS, *["-D" + x for x in defines], "-save-temps", "-c", os.path.join(CSRC, src),
                   "-o", obj]
            if resource_usage:
                cmd.insert(1, "-Rpass-analysis=kernel-resource-usage")
            r = subprocess.run(cmd, capture_output=True, text=True, cwd=work)
            if r.returncode != 0:
                raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
            return obj, r.stderr, device_asm_path(work, src)

        with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 1)) as ex:
            results = list(ex.map(compile_one, SOURCES))
        for _, err, _ in results:
            if verbose and err.strip():
                print(err, file=sys.stderr)
        if check_waits:
            bad = []
            for src, (_, _, asm) in zip(SOURCES, results):
                with open(asm) as f:
                    viol, _ = waitstates.scan(f.read())
                bad += [f"{src}: {v}" for v in viol]
            if bad:
                raise RuntimeError("inline-asm wait states violated:\n" + "\n".join(bad[:20]))
        out_tmp = out + ".tmp"
        cmd = [cc, "--offload-arch=gfx950", "-shared", "-fPIC", *[o for o, _, _ in results], "-o", out_tmp]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"link failed:\n{r.stderr}")
        os.replace(out_tmp, out)
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return out


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("--resource-usage", action="store_true")
    ap.add_argument("-D", dest="defines", action="append", default=[], help="extra preprocessor define")
    ap.add_argument("-o", dest="out", default=LIB)
    a = ap.parse_args()
    print(build(verbose=a.verbose or a.resource_usage, resource_usage=a.resource_usage, defines=a.defines, out=a.out))
